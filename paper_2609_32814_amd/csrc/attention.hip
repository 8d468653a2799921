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

constexpr int kFwdThreads = 256;  // 4 wavefronts
constexpr int kQRows = 32;        // query rows per wave
constexpr int kBlockRows = 128;   // query rows per workgroup
constexpr int kKeys = 32;         // keys per block

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

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return static_cast<uint32_t>(f32_to_bf16(a)) | (static_cast<uint32_t>(f32_to_bf16(b)) << 16);
}
__device__ __forceinline__ uint32_t pair16(short lo, short hi) {
  return static_cast<uint16_t>(lo) | (static_cast<uint32_t>(static_cast<uint16_t>(hi)) << 16);
}

// Value block in LDS: 32 key rows of DH bf16; the 16-byte chunk c of row r
// sits at chunk c ^ 2 (r & 3), so the 4 rows of a transposing read fall on
// distinct banks.
template <int DH>
__device__ __forceinline__ int vrow_off(int r, int c) {
  return r * (DH * 2) + ((c ^ (2 * (r & 3))) << 4);
}

template <int DH>
__global__ __launch_bounds__(kFwdThreads) void attn_fwd_kernel(const AttnParams p) {
  constexpr int NCH = DH / 32;  // 32-feature output chunks
  constexpr int KS = DH / 16;   // 16-feature contraction steps over a head
  constexpr int CPR = DH / 8;   // 16-byte chunks per row
  constexpr int RPC = 64 / CPR; // rows per 1 KB copy
  __shared__ __attribute__((aligned(16))) char vblk[kKeys * DH * 2];
  __shared__ int32_t kpos_s[kKeys];
  __shared__ int32_t qpos_s[kBlockRows];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 31, lh = lane >> 5;
  const int q = p.q, m = DH / q;

  // ---- work item.  Consecutive workgroups take the same block level of
  // different (sequence, head) pairs, and the latest (longest) query blocks
  // of every type come first.
  const int32_t BH = p.B * p.n_heads;
  const int32_t bh = blockIdx.x % BH;
  int32_t r = blockIdx.x / BH;
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

  if (threadIdx.x < kBlockRows) {
    const int32_t pos = q0 + threadIdx.x;
    qpos_s[threadIdx.x] = pos < qend ? p.perm[pos] : -1;
  }
  __syncthreads();
  // positions increase along the block: the workgroup's last query, and the
  // wave's first and last
  const int32_t nvalid = min(kBlockRows, qend - q0);
  const int32_t wg_last = qpos_s[nvalid - 1];
  const int32_t wv = min(kQRows, nvalid - wave * kQRows);  // valid rows of this wave (may be <= 0)
  const int32_t wave_first = wv > 0 ? qpos_s[wave * kQRows] : 0x7fffffff;
  const int32_t wave_last = wv > 0 ? qpos_s[wave * kQRows + wv - 1] : -1;

  // the wave's query rows as the B operand: lane half lh holds features
  // 16 ks + 8 lh .. + 7 of row lr for every step ks
  const int32_t my_qpos = qpos_s[wave * kQRows + lr];
  uint4 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qf[ks] = make_uint4(0, 0, 0, 0);
    if (my_qpos >= 0) qf[ks] = *reinterpret_cast<const uint4*>(Qg + static_cast<int64_t>(my_qpos) * ldq + 16 * ks + 8 * lh);
  }

  // online softmax state of the lane's query (shared with lane l ^ 32)
  float run_max = -INFINITY, run_sum = 0.f;
  f32x16_t acc[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;

  for (int j = 0; j < q; ++j) {
    const uint32_t fmask = attn_fmask(p.law, q, i, j);
    const float scale = kLog2e * __builtin_amdgcn_rsqf(static_cast<float>(__popc(fmask) * m));
    const int32_t k_lo = p.offsets[j], k_hi = p.offsets[j + 1];
    for (int32_t k0 = k_lo; k0 < k_hi; k0 += kKeys) {
      if (threadIdx.x < kKeys) kpos_s[threadIdx.x] = k0 + static_cast<int32_t>(threadIdx.x) < k_hi ? p.perm[k0 + threadIdx.x] : 0x7fffffff;
      __syncthreads();
      const int32_t first = kpos_s[0];
      if (first > wg_last) {  // this block and the rest of type j follow every query
        __syncthreads();
        break;
      }
      // the value block into LDS (rows past the type's end copy zeros)
      for (int cb = wave; cb < kKeys / RPC; cb += 4) {
        const int row = cb * RPC + lane / CPR;
        const int c = (lane % CPR) ^ (2 * (row & 3));
        const int32_t kp = kpos_s[row];
        const void* g = kp < p.S ? static_cast<const void*>(Vg + static_cast<int64_t>(kp) * ldk + 8 * c)
                                 : static_cast<const void*>(g_attn_zero);
        dma16(g, lds_addr(vblk + cb * 1024));
      }
      const bool active = first <= wave_last;  // some key of the block precedes a query of the wave
      float s[16];
      if (active) {
        const int32_t kp = kpos_s[lr];
        const uint16_t* kr = Kg + static_cast<int64_t>(kp < p.S ? kp : 0) * ldk;
        f32x16_t sa;
#pragma unroll
        for (int e = 0; e < 16; ++e) sa[e] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int a0 = (16 * ks) / m, a1 = (16 * ks + 15) / m;
          if (!(((fmask >> a0) | (fmask >> a1)) & 1u)) continue;
          const int al = (16 * ks + 8 * lh) / m;
          uint4 kf = make_uint4(0, 0, 0, 0);
          if ((fmask >> al) & 1u) kf = *reinterpret_cast<const uint4*>(kr + 16 * ks + 8 * lh);
          sa = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, kf),
                                                        __builtin_bit_cast(bf16x8_t, qf[ks]), sa, 0, 0, 0);
        }
        // lane holds query lr against keys 8 (e / 4) + 4 lh + e % 4
        const bool full = kpos_s[kKeys - 1] <= wave_first;  // no key of the block follows a query of the wave
        float bmax = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kk = 8 * (e / 4) + 4 * lh + (e % 4);
          float v = sa[e] * scale;
          if (!full && kpos_s[kk] > my_qpos) v = -INFINITY;
          s[e] = v;
          bmax = fmaxf(bmax, v);
        }
        bmax = fmaxf(bmax, __shfl_xor(bmax, 32));
        const float new_max = fmaxf(run_max, bmax);
        // a row whose keys so far are all masked keeps max -inf and zero
        // probabilities
        const bool none = new_max == -INFINITY;
        const float corr = none ? 1.f : __builtin_amdgcn_exp2f(run_max - new_max);
        float bsum = 0.f;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float pe = none ? 0.f : __builtin_amdgcn_exp2f(s[e] - new_max);
          s[e] = pe;
          bsum += pe;
        }
        bsum += __shfl_xor(bsum, 32);
        run_sum = run_sum * corr + bsum;
        run_max = new_max;
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[c][e] *= corr;
      }
      wait_vm_all();
      __syncthreads();  // the value block has landed
      if (active) {
        // O^T += V^T P^T in two 16-key steps: step kk takes the lane's
        // probabilities e = 8 kk .. 8 kk + 7, the keys 16 kk + 4 lh + 0..3
        // and 16 kk + 8 + 4 lh + 0..3
        const int g = lane >> 4, pp = lane & 15;
        const int rr = pp >> 2, qq = pp & 3;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          uint4 pf;
          pf.x = pack_bf16(s[8 * kk + 0], s[8 * kk + 1]);
          pf.y = pack_bf16(s[8 * kk + 2], s[8 * kk + 3]);
          pf.z = pack_bf16(s[8 * kk + 4], s[8 * kk + 5]);
          pf.w = pack_bf16(s[8 * kk + 6], s[8 * kk + 7]);
          const int row0 = 16 * kk + 4 * (g >> 1) + rr;
#pragma unroll
          for (int c = 0; c < NCH; ++c) {
            // in 16-lane group g, lanes 4 rr + qq address features
            // f .. f + 3 of key rows row0 and row0 + 8; lane pp receives
            // feature 32 c + 16 (g & 1) + pp of those 4 + 4 rows
            const int f = 32 * c + 16 * (g & 1) + 4 * qq;
            const char* a0 = vblk + vrow_off<DH>(row0, f >> 3) + ((f >> 2) & 1) * 8;
            const char* a1 = vblk + vrow_off<DH>(row0 + 8, f >> 3) + ((f >> 2) & 1) * 8;
            const v4i16_t w0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a0));
            const v4i16_t w1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(a1));
            uint4 vf;
            vf.x = pair16(w0[0], w0[1]);
            vf.y = pair16(w0[2], w0[3]);
            vf.z = pair16(w1[0], w1[1]);
            vf.w = pair16(w1[2], w1[3]);
            acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vf),
                                                             __builtin_bit_cast(bf16x8_t, pf), acc[c], 0, 0, 0);
          }
        }
      }
      __syncthreads();  // every wave is done with the value block and the key positions
    }
  }

  // ---- O = acc / sum: lane holds query lr, features 32 c + 8 a + 4 lh + 0..3
  if (my_qpos >= 0) {
    const float inv = run_sum > 0.f ? 1.f / run_sum : 0.f;
    const int64_t o = (static_cast<int64_t>(b) * p.S + my_qpos) * ldq + h * DH;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int f = 32 * c + 8 * a + 4 * lh;
        const float v0 = acc[c][4 * a] * inv, v1 = acc[c][4 * a + 1] * inv;
        const float v2 = acc[c][4 * a + 2] * inv, v3 = acc[c][4 * a + 3] * inv;
        if (p.odtype == 0) {
          *reinterpret_cast<float4*>(static_cast<float*>(p.O) + o + f) = make_float4(v0, v1, v2, v3);
        } else {
          *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.O) + o + f) = make_uint2(pack_bf16(v0, v1), pack_bf16(v2, v3));
        }
      }
    if (p.lse && lh == 0) {
      const float l = run_sum > 0.f ? (run_max + __log2f(run_sum)) * 0.6931471805599453f : -INFINITY;
      p.lse[(static_cast<int64_t>(b) * p.n_heads + h) * p.S + my_qpos] = l;
    }
  }
}

// ---- decode ---------------------------------------------------------------------

constexpr int kDecThreads = 256;
constexpr int kDecKeysPerTeam = 4;

template <int DH>
constexpr int dec_chunk() { return kDecKeysPerTeam * (kDecThreads / (DH / 8)); }
template <int DH>
constexpr int dec_smem_max() { return static_cast<int>(sizeof(float)) * (kDecThreads / (DH / 8)) * kAttnDecHeads * DH; }

// One chunk of the cache of one sequence against up to kAttnDecHeads query
// heads that share one key/value head.
template <int DH>
__global__ __launch_bounds__(kDecThreads) void attn_decode_part_kernel(const AttnParams p) {
  constexpr int T = DH / 8;            // lanes per key
  constexpr int NT = kDecThreads / T;  // teams
  constexpr int CH = dec_chunk<DH>();  // keys per chunk
  constexpr int G = kAttnDecHeads;
  extern __shared__ __attribute__((aligned(16))) float dsm[];  // [NT][gh][DH] team partial outputs
  __shared__ float sc[G][CH];          // scores, then probabilities
  __shared__ uint32_t fm_s[32];        // F(i, j) as a bit mask, per key type j
  __shared__ float ml_s[G][2];

  const int chunk = blockIdx.x;
  const int hk = blockIdx.y / p.head_groups, hg = blockIdx.y % p.head_groups;
  const int b = blockIdx.z;
  const int g_all = p.n_heads / p.n_kv;
  const int h0 = hk * g_all + hg * G;
  const int gh = min(G, g_all - hg * G);
  const int q = p.q, m = DH / q;
  const int32_t L = min(p.cache_len[b], p.S);
  const int32_t u0 = chunk * CH;
  if (L <= 0 || u0 >= L) return;
  const int i = p.pos_type[L - 1];
  if (static_cast<unsigned>(i) >= static_cast<unsigned>(q)) return;  // the merge writes zeros
  const int32_t u1 = min(L, u0 + CH);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int team = tid / T, t = tid % T;
  if (tid < q) fm_s[tid] = attn_fmask(p.law, q, i, tid);

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

  // ---- scores of the team's keys u0 + team + NT k
  int32_t jt[kDecKeysPerTeam];
  uint4 kv[kDecKeysPerTeam];
#pragma unroll
  for (int k = 0; k < kDecKeysPerTeam; ++k) {
    const int32_t u = u0 + team + NT * k;
    jt[k] = u < u1 ? p.pos_type[u] : -1;
    const bool key_ok = static_cast<unsigned>(jt[k]) < static_cast<unsigned>(q);
    kv[k] = make_uint4(0, 0, 0, 0);
    if (key_ok && ((fm_s[key_ok ? jt[k] : 0] >> al) & 1u)) kv[k] = *reinterpret_cast<const uint4*>(Kc + static_cast<int64_t>(u) * ldk);
  }
#pragma unroll
  for (int k = 0; k < kDecKeysPerTeam; ++k) {
    const uint32_t w[4] = {kv[k].x, kv[k].y, kv[k].z, kv[k].w};
    float kf[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      kf[2 * e] = bf16_to_f32(w[e] & 0xffffu);
      kf[2 * e + 1] = bf16_to_f32(w[e] >> 16);
    }
    float d[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
      float a = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) a += qf[hh][e] * kf[e];
      d[hh] = a;
    }
#pragma unroll
    for (int o = T / 2; o > 0; o >>= 1)
#pragma unroll
      for (int hh = 0; hh < G; ++hh) d[hh] += __shfl_xor(d[hh], o, T);
    const int32_t u = u0 + team + NT * k;
    if (t == 0 && u < u1) {
      const bool key_ok = static_cast<unsigned>(jt[k]) < static_cast<unsigned>(q);
      const float scale = key_ok ? kLog2e * __builtin_amdgcn_rsqf(static_cast<float>(__popc(fm_s[jt[k]]) * m)) : 0.f;
#pragma unroll
      for (int hh = 0; hh < G; ++hh) sc[hh][u - u0] = key_ok ? d[hh] * scale : -INFINITY;
    }
  }
  __syncthreads();

  // ---- the chunk's softmax, one wave per head
  const int32_t n = u1 - u0;
  for (int hh = wave; hh < gh; hh += kDecThreads / 64) {
    float mx = -INFINITY;
    for (int32_t u = lane; u < n; u += 64) mx = fmaxf(mx, sc[hh][u]);
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    float sum = 0.f;
    for (int32_t u = lane; u < n; u += 64) {
      const float e = mx == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sc[hh][u] - mx);
      sc[hh][u] = e;
      sum += e;
    }
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if (lane == 0) {
      ml_s[hh][0] = mx;
      ml_s[hh][1] = sum;
    }
  }
  __syncthreads();

  // ---- the team's weighted value rows, then the teams summed in order
  uint4 vv[kDecKeysPerTeam];
#pragma unroll
  for (int k = 0; k < kDecKeysPerTeam; ++k) {
    const int32_t u = u0 + team + NT * k;
    vv[k] = make_uint4(0, 0, 0, 0);
    if (u < u1) vv[k] = *reinterpret_cast<const uint4*>(Vc + static_cast<int64_t>(u) * ldk);
  }
  float o[G][8];
#pragma unroll
  for (int hh = 0; hh < G; ++hh)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[hh][e] = 0.f;
#pragma unroll
  for (int k = 0; k < kDecKeysPerTeam; ++k) {
    const int32_t u = u0 + team + NT * k;
    if (u >= u1) continue;
    const uint32_t w[4] = {vv[k].x, vv[k].y, vv[k].z, vv[k].w};
    float vf[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      vf[2 * e] = bf16_to_f32(w[e] & 0xffffu);
      vf[2 * e + 1] = bf16_to_f32(w[e] >> 16);
    }
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
      const float pw = hh < gh ? sc[hh][u - u0] : 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[hh][e] += pw * vf[e];
    }
  }
#pragma unroll
  for (int hh = 0; hh < G; ++hh) {
    if (hh >= gh) break;
    float* dst = dsm + (static_cast<int64_t>(team) * gh + hh) * DH + 8 * t;
    *reinterpret_cast<float4*>(dst) = make_float4(o[hh][0], o[hh][1], o[hh][2], o[hh][3]);
    *reinterpret_cast<float4*>(dst + 4) = make_float4(o[hh][4], o[hh][5], o[hh][6], o[hh][7]);
  }
  __syncthreads();
  const int64_t slot0 = (static_cast<int64_t>(b) * p.n_heads + h0) * p.nchunks + chunk;
  for (int x = tid; x < gh * DH; x += kDecThreads) {
    const int hh = x / DH, f = x % DH;
    float a = 0.f;
    for (int tm = 0; tm < NT; ++tm) a += dsm[(tm * gh + hh) * DH + f];
    p.part_o[(slot0 + static_cast<int64_t>(hh) * p.nchunks) * DH + f] = a;
  }
  if (tid < gh) {
    const int64_t s = slot0 + static_cast<int64_t>(tid) * p.nchunks;
    p.part_ml[2 * s] = ml_s[tid][0];
    p.part_ml[2 * s + 1] = ml_s[tid][1];
  }
}

// Merges the chunks of one (sequence, head): O = sum_c 2^(m_c - M) o_c /
// sum_c 2^(m_c - M) l_c with M the largest chunk maximum.
template <int DH>
__global__ __launch_bounds__(DH) void attn_decode_merge_kernel(const AttnParams p) {
  constexpr int CH = dec_chunk<DH>();
  const int b = blockIdx.x / p.n_heads, h = blockIdx.x % p.n_heads;
  const int f = threadIdx.x;
  const int32_t L = min(p.cache_len[b], p.S);
  float v = 0.f;
  const bool ok = L > 0 && static_cast<unsigned>(p.pos_type[L - 1]) < static_cast<unsigned>(p.q);
  if (ok) {
    const int32_t nch = (L + CH - 1) / CH;
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

template <int DH>
hipError_t launch_decode_dh(const AttnParams& p, hipStream_t stream) {
  constexpr int T = DH / 8;
  const int gmax = std::min(kAttnDecHeads, p.n_heads / p.n_kv);
  const size_t smem = sizeof(float) * static_cast<size_t>(kDecThreads / T) * gmax * DH;
  static std::atomic<unsigned long long> set{0};
  hipError_t e = ensure_lds_limit(reinterpret_cast<const void*>(attn_decode_part_kernel<DH>), set, dec_smem_max<DH>());
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_decode_part_kernel<DH>, dim3(p.nchunks, p.n_kv * p.head_groups, p.B), dim3(kDecThreads), smem,
                     stream, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_decode_merge_kernel<DH>, dim3(p.B * p.n_heads), dim3(DH), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_fwd(const AttnParams& p, hipStream_t stream) {
  const int64_t grid = static_cast<int64_t>(p.B) * p.n_heads * p.items_per_bh;
  if (grid <= 0 || grid > 0x7fffffff) return hipErrorInvalidValue;
  switch (p.head_dim) {
    case 64: hipLaunchKernelGGL(attn_fwd_kernel<64>, dim3(static_cast<unsigned>(grid)), dim3(kFwdThreads), 0, stream, p); break;
    case 128: hipLaunchKernelGGL(attn_fwd_kernel<128>, dim3(static_cast<unsigned>(grid)), dim3(kFwdThreads), 0, stream, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int32_t attn_decode_chunk(int32_t head_dim) {
  return head_dim == 64 ? dec_chunk<64>() : head_dim == 128 ? dec_chunk<128>() : 0;
}

hipError_t launch_attn_decode(const AttnParams& p, hipStream_t stream) {
  switch (p.head_dim) {
    case 64: return launch_decode_dh<64>(p, stream);
    case 128: return launch_decode_dh<128>(p, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace starq
