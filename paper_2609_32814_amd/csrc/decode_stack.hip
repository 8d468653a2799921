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
// partial sums) is otherwise written with agent-coherent stores and read with
// agent-coherent loads (copies into LDS with sc1), so no cache
// write-back or invalidate is needed; arrival counters are agent-scope
// atomics that only grow (a layer's target is a multiple of the item
// count).  An all-workgroup arrival is spread over kSubCounters counters,
// each on its own 256-byte line, and a waiter sums them with one vector
// load: many workgroups adding to one address serialise at the memory
// side, which on this part costs more than the extra lanes of the poll.
// The slice plan of an item depends only on the row types, so it is made
// once per launch; each layer only issues the copies.
//
// Summing the down chunks, in chunk order either way, so results do not
// depend on timing: for a few rows (RES kernels) every workgroup keeps the
// running state h in LDS and, in the next layer, sums the chunks itself
// into its copy of h and into the next up input; for more rows the chunks
// of one tile are summed by whichever of its workgroups arrives last, which
// writes h and the next input for everyone (three hand-offs per layer).
//
// RES kernels hand H and the down chunks over as tagged 64-bit words (the
// data and the writing layer plus one, stored and loaded whole): a reader
// polls the words it needs until they carry the layer it waits for, so
// the wait and the data read are one load, and a writer neither waits for
// its stores to land nor bumps a counter.  The down chunks alternate
// between two buffers by layer parity; every workgroup owns a down item
// and reads all chunks of a layer before it writes its own of the next, so
// no chunk is overwritten before every workgroup has read it.  Every wait
// is bounded: after about half a second of spinning the kernel raises the
// error flag (the first word of the workspace, which star_decode_status
// reads) and carries on, so it always terminates; a wait that finds the
// flag raised gives up at once, so a lost step ends after one bound, not
// one per wait.
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
constexpr int kFlagPoll = 255;       // a waiter reads the error flag every 256 spins

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

// Tagged hand-off words: the data in the low half, the writing layer plus
// one in the high half, stored and loaded whole (single-copy atomic), so a
// reader that sees the tag it waits for has the data with it.
__device__ __forceinline__ void st_tagged(uint64_t* p, uint32_t v, uint32_t tag) {
  __hip_atomic_store(p, (static_cast<uint64_t>(tag) << 32) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_tagged(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Settles n words at once: reloads every word that does not yet carry tag,
// all together, until none is left, so the wait ends one round trip after
// the last word lands however many of them came late.  Slots with
// src[i] == nullptr are ignored.  After about half a second it raises the error flag
// and gives up.
template <int N>
__device__ __forceinline__ void settle_all(const uint64_t* const (&src)[N], uint64_t (&w)[N], uint32_t tag,
                                           int32_t* err) {
  int spins = 0;
  while (true) {
    bool done = true;
#pragma unroll
    for (int i = 0; i < N; ++i) done &= src[i] == nullptr || static_cast<uint32_t>(w[i] >> 32) == tag;
    if (done) break;
    __builtin_amdgcn_s_sleep(1);
    if (++spins > kSpinLimit) {
      st_agent(reinterpret_cast<uint32_t*>(err), 1u);
      break;
    }
    // once some wait has timed out the step is lost: stop waiting at once
    if ((spins & kFlagPoll) == 0 && ld_agent(reinterpret_cast<const uint32_t*>(err)) != 0u) break;
#pragma unroll
    for (int i = 0; i < N; ++i)
      if (src[i] != nullptr && static_cast<uint32_t>(w[i] >> 32) != tag) w[i] = ld_tagged(src[i]);
  }
}

// k in B(i, j): law 0 {i, j}; law 1 every group; law 2 (tensor power of
// the two-group law) every bit of k equal to that bit of i or of j; law 3
// (graph algebra, bit j of adj[i] for the edge i -> j) {i} for j = i, {i, j}
// for an edge, nothing otherwise
__device__ __forceinline__ bool in_support(int law, const uint64_t* adj, int i, int j, int k) {
  if (law == 2) return ((k ^ i) & (k ^ j)) == 0;
  if (law == 3) {
    // graph algebra: B(i,i) = {i}, B(i,j) = {i, j} for an edge i -> j, empty otherwise
    if (j == i) return k == i;
    return ((adj[i] >> j) & 1ull) && (k == i || k == j);
  }
  return law == 1 || k == i || k == j;
}
// the input group of index x: the last g with starts[g] <= x, by binary
// search over the starts (held in LDS: searched from the kernel's argument
// block, every step was a dependent scalar load)
__device__ __forceinline__ int group_of(const int32_t* starts, int q, int32_t x) {
  int lo = 0, hi = q - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (x >= starts[mid]) lo = mid;
    else hi = mid - 1;
  }
  return lo;
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

// MB: 16-row blocks of the step (M <= 16 MB).  RES: the running state h is
// kept in every workgroup's LDS (small M only), H and the down chunks travel
// as tagged words, and the next layer's up items sum the chunks themselves,
// so a layer needs two hand-offs instead of three; in the last layer each
// down tile's first chunk sums the tile's chunks to write Y.
template <int MB, bool RES>
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
  const int kmax = (max(p.D, p.kc) + 127) & ~127;
  constexpr int NOFF = kMaxSlices / 4;  // slices per wave and slot
  // staging writes whole 1 KB copies, so round the x buffer up to 1 KB
  const int xbytes = max((M * kmax * 2 + 1023) & ~1023, kRedBytes);
  char* xbuf = lds;
  // slots: 0 up weights, 1 down weights, 2 (gated FFN) gate weights; the
  // gate item is the up item, so slot 2 shares slot 0's slice plan
  const int nslots = p.gated ? 3 : 2;
  char* slot_base[3] = {lds + xbytes, lds + xbytes + (kmax / SLICE) * 1024,
                        lds + xbytes + 2 * (kmax / SLICE) * 1024};
  // RES: the running state [M][D] fp32
  float* hres = reinterpret_cast<float*>(lds + xbytes + nslots * (kmax / SLICE) * 1024);
  int32_t* err = p.err;
  int32_t* cnt_up = p.cnt + kCounterStride;
  int32_t* cnt_dn = cnt_up + kCounterStride * kSubCounters;
  int32_t* tile_cnt = cnt_dn + kCounterStride * kSubCounters;  // one line per down tile
  const void* zero = g_stack_zero;

  const Item iu = up_item(p);
  const Item idn = down_item(p);

  // Which rows need input group g for output group j (one ballot per
  // group by wave 0), then the needed slices of [k_lo, k_hi) in K order and
  // the rows each 8-wide piece of them serves.
  auto plan = [&](int slot, const Item& it, const int32_t* KS) {
    if (wave == 0) {
      // a row whose type lies outside [0, q) has an empty support
      const int t = lane < M ? p.types[lane] : -1;
      const bool valid = t >= 0 && t < p.q;
      for (int g = 0; g < p.q; ++g) {
        const unsigned long long m = __ballot(valid && in_support(p.law, p.adj, t, it.j, g));
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
    __syncthreads();
  };

  // Element offsets into W of this lane's 16 bytes of slice wave + 4 t of a
  // slot, computed once: the per-layer copies then issue without waiting on
  // LDS.  Slices past the plan get offset -1.
  auto copy_offsets = [&](int slot, const Item& it, int32_t ldw, int32_t (&off)[NOFF]) {
    const int ns_ = nslices_s[slot];
#pragma unroll
    for (int t = 0; t < NOFF; ++t) {
      const int i = wave + 4 * t;
      off[t] = -1;
      if (i < ns_) {
        int32_t row = it.k_lo + slices_s[slot][i] * SLICE + (lane >> 1);
        row = row < it.k_hi ? row : it.k_hi - 1;  // finite filler, its inputs are zero
        int32_t col = it.n0 + 8 * (lane & 1);
        col = col < it.nend ? col : it.n0;
        off[t] = row * ldw + col;
      }
    }
  };
  auto copy = [&](int slot, const uint16_t* W, const int32_t (&off)[NOFF]) {
    char* sb = slot_base[slot];
#pragma unroll
    for (int t = 0; t < NOFF; ++t)
      if (off[t] >= 0) dma16(W + off[t], lds_addr(sb + (wave + 4 * t) * 1024));
  };

  // Arrival on this workgroup's sub-counter of a set, and a bounded wait
  // until the set's sum reaches target (wave 0 polls, the others wait at
  // the barrier).
  auto arrive = [&](int32_t* set) {
    __hip_atomic_fetch_add(set + kCounterStride * (blockIdx.x % kSubCounters), 1, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
  };
  auto wait_for = [&](int32_t* set, int32_t target) {
    if (wave == 0) {
      int spins = 0;
      while (true) {
        int32_t v = lane < kSubCounters
                        ? static_cast<int32_t>(ld_agent(reinterpret_cast<uint32_t*>(set + kCounterStride * lane)))
                        : 0;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
        if (v >= target) break;
        __builtin_amdgcn_s_sleep(1);
        if (++spins > kSpinLimit) {
          if (lane == 0) st_agent(reinterpret_cast<uint32_t*>(err), 1u);
          break;
        }
        if ((spins & kFlagPoll) == 0 && ld_agent(reinterpret_cast<const uint32_t*>(err)) != 0u) break;
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

  // RES, layer l >= 1: h_l = sum of the down chunks of layer l - 1 (chunk
  // order) + bias (+ h_{l-1}), kept in hres and written as the swizzled bf16
  // up input (K = D, padded to a multiple of 128 with zeros).  The chunks
  // are tagged words (tag l, buffer (l - 1) & 1), polled in place: the wait
  // for the other workgroups and the read of their data are one load.  Each
  // thread takes four consecutive columns of one row.
  auto stage_resident = [&](int l) {
    __syncthreads();  // every wave is done with the x buffer
    const int kx = (p.D + 127) & ~127;
    const int quads = kx / 4;
    const float* b = p.bd[l - 1];
    const uint32_t tag = static_cast<uint32_t>(l);
    const uint64_t* tp = p.tpart + static_cast<int64_t>((l - 1) & 1) * p.ns * M * p.D;
    for (int e = tid; e < M * quads; e += kThreads) {
      const int m = e / quads;
      const int k = 4 * (e - m * quads);
      uint2 packed = make_uint2(0u, 0u);
      if (k < p.D) {
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        for (int c0 = 0; c0 < p.ns; c0 += 4) {
          uint64_t w[16];
          const uint64_t* src[16];
#pragma unroll
          for (int cc = 0; cc < 4; ++cc) {
            const uint64_t* base = tp + (static_cast<int64_t>(min(c0 + cc, p.ns - 1)) * M + m) * p.D + k;
#pragma unroll
            for (int x = 0; x < 4; ++x) {
              src[4 * cc + x] = c0 + cc < p.ns ? base + x : nullptr;
              w[4 * cc + x] = c0 + cc < p.ns ? ld_tagged(base + x) : 0ull;
            }
          }
          settle_all(src, w, tag, err);
#pragma unroll
          for (int cc = 0; cc < 4; ++cc) {
            if (c0 + cc < p.ns) {
#pragma unroll
              for (int x = 0; x < 4; ++x) v[x] += __uint_as_float(static_cast<uint32_t>(w[4 * cc + x]));
            }
          }
        }
        if (b) {
          const float4 bv = *reinterpret_cast<const float4*>(b + k);
          v[0] += bv.x; v[1] += bv.y; v[2] += bv.z; v[3] += bv.w;
        }
        float* hr = hres + m * p.D + k;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          if (p.residual) v[x] += hr[x];
          hr[x] = v[x];
        }
        packed.x = f32_to_bf16(v[0]) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
        packed.y = f32_to_bf16(v[2]) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
      }
      const int c = (k >> 3) ^ (m & 15);
      *reinterpret_cast<uint2*>(xbuf + (m * kx + 8 * c + (k & 7)) * 2) = packed;
    }
    wait_vm_all();  // the weight copies issued before
    __syncthreads();
  };

  // RES: the down item's slice of H (tagged bf16 pairs of layer l, tag
  // l + 1) polled in place into the swizzled x buffer; inputs past k_hi are
  // zero.
  auto stage_h = [&](const Item& it, uint32_t tag) {
    __syncthreads();  // every wave is done with the x buffer
    const int kx = (it.k_hi - it.k_lo + 127) & ~127;
    const int pairs = kx / 2;
    const int total = M * pairs;
    const int64_t ldh = p.F / 2;
    for (int e0 = tid; e0 < total; e0 += 4 * kThreads) {
      uint64_t w[4];
      const uint64_t* src[4];
      bool ok[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int e = e0 + r * kThreads;
        const int m = min(e / pairs, M - 1);
        const int k = it.k_lo + 2 * (e - (e / pairs) * pairs);
        ok[r] = e < total && k < it.k_hi;
        src[r] = ok[r] ? p.tH + m * ldh + k / 2 : nullptr;
        w[r] = ok[r] ? ld_tagged(src[r]) : 0ull;
      }
      settle_all(src, w, tag, err);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int e = e0 + r * kThreads;
        if (e < total) {
          const int m = e / pairs;
          const int kr = 2 * (e - m * pairs);
          const uint32_t v = ok[r] ? static_cast<uint32_t>(w[r]) : 0u;
          const int c = (kr >> 3) ^ (m & 15);
          *reinterpret_cast<uint32_t*>(xbuf + (m * kx + 8 * c + (kr & 7)) * 2) = v;
        }
      }
    }
    wait_vm_all();  // the weight copies issued before
    __syncthreads();
  };

  // acc over the item's slices; lane group G = lane / 16 holds K rows
  // 8G..8G+7 of a slice for column n0 + lane % 16, and rows 16 mb + lane % 16.
  // A wave's slices are wave, wave + 4, ...; RB of them have their LDS reads
  // in flight together.
  constexpr int RB = MB == 1 ? 8 : (MB == 2 ? 4 : 2);
  // (slot: the slice plan; data_slot: where the weights are)
  auto compute = [&](int slot, int data_slot, const Item& it, f32x4_t (&acc)[MB]) {
    const int G = lane >> 4;
    const int pl = lane & 15;
    const int kx = (it.k_hi - it.k_lo + 127) & ~127;
    const int ns_ = nslices_s[slot];
    const char* sb = slot_base[data_slot];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int t0 = 0; wave + 4 * t0 < ns_; t0 += RB) {
      uint4 wf[RB], xv[RB][MB];
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        const int i = wave + 4 * (t0 + r);
        if (i < ns_) {
          const char* base = sb + i * 1024 + (8 * G + (pl >> 2)) * 32 + (pl & 3) * 8;
          const v4i16_t w0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(base));
          const v4i16_t w1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((STARQ_LDS v4i16_t*)(base + 128));
          wf[r].x = static_cast<uint16_t>(w0[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[1])) << 16);
          wf[r].y = static_cast<uint16_t>(w0[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w0[3])) << 16);
          wf[r].z = static_cast<uint16_t>(w1[0]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[1])) << 16);
          wf[r].w = static_cast<uint16_t>(w1[2]) | (static_cast<uint32_t>(static_cast<uint16_t>(w1[3])) << 16);
          const int32_t krel = slices_s[slot][i] * SLICE + 8 * G;
          const unsigned long long gm = pmask_s[slot][i][G];
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) {
            const int m = 16 * mb + pl;
            const int mr = min(m, M - 1);  // rows past M read row M - 1, then zero
            const int c = (krel >> 3) ^ (mr & 15);
            xv[r][mb] = *reinterpret_cast<const uint4*>(xbuf + (mr * kx + 8 * c) * 2);
            if (!(m < M && ((gm >> m) & 1ull))) xv[r][mb] = make_uint4(0, 0, 0, 0);
          }
        }
      }
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        if (wave + 4 * (t0 + r) < ns_) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
            // D[n][m] += W^T x^T: the lane ends with 4 consecutive columns of row m
            acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, wf[r]),
                                                              __builtin_bit_cast(bf16x8_t, xv[r][mb]),
                                                              acc[mb], 0, 0, 0);
        }
      }
    }
  };

  // Fixed-order sum of the four waves' partials (through LDS, reusing the
  // x buffer); thread tid then owns rows 16 mb + l % 16, columns
  // n0 + 4 (l / 16) .. + 3 with mb = tid / 64, l = tid % 64 (mb < MB).
  auto reduce = [&](f32x4_t (&acc)[MB], f32x4_t& z) {
    __syncthreads();  // every wave is done with the x buffer
    f32x4_t* red = reinterpret_cast<f32x4_t*>(xbuf);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) red[(wave * 4 + mb) * 64 + lane] = acc[mb];
    __syncthreads();
    const int mb = tid >> 6;
    z = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (mb < MB) {
      z = red[(0 * 4 + mb) * 64 + lane];
      z += red[(1 * 4 + mb) * 64 + lane];
      z += red[(2 * 4 + mb) * 64 + lane];
      z += red[(3 * 4 + mb) * 64 + lane];
    }
  };

  const int my_m = 16 * (tid >> 6) + (lane & 15);
  const int my_dn = 4 * (lane >> 4);

  // prologue: slice plans and copy offsets, then the weights of layer 0
  // (the group starts searched from LDS)
  __shared__ int32_t SD_s[kMaxQGroups + 1], SF_s[kMaxQGroups + 1];
  for (int i = tid; i <= p.q; i += kThreads) {
    SD_s[i] = p.SD[i];
    SF_s[i] = p.SF[i];
  }
  __syncthreads();
  int32_t off_u[NOFF], off_d[NOFF];
  if (iu.valid) plan(0, iu, SD_s);
  if (idn.valid) plan(1, idn, SF_s);
  if (iu.valid) copy_offsets(0, iu, p.F, off_u);
  if (idn.valid) copy_offsets(1, idn, p.D, off_d);
  if (iu.valid) copy(0, p.Wu[0], off_u);
  if (iu.valid && p.gated) copy(2, p.Wg[0], off_u);
  if (idn.valid) copy(1, p.Wd[0], off_d);
  if (RES) {
    for (int e = tid; e < M * p.D; e += kThreads) hres[e] = bf16_to_f32(p.X[e]);
  }

  for (int l = 0; l < p.L; ++l) {
    const bool last = l + 1 == p.L;
    // ---------------- up projection: H = act(x W_up + b_up) ----------------
    if (l > 0) {
      if (RES)
        stage_resident(l);
      else
        wait_for(cnt_dn, p.nt_dn * l);
    }
    if (iu.valid) {
      if (!RES || l == 0) {
        const uint16_t* xin = (l == 0) ? p.X : p.hb + static_cast<int64_t>(l & 1) * M * p.D;
        stage_x(iu, xin, p.D);
        wait_vm_all();
        __syncthreads();
      }
      // both products first: the cross-wave sums reuse the x buffer
      f32x4_t acc[MB], accg[MB], z, zg = f32x4_t{0.f, 0.f, 0.f, 0.f};
      if (p.gated) compute(0, 2, iu, accg);
      compute(0, 0, iu, acc);
      if (p.gated) reduce(accg, zg);
      reduce(acc, z);
      const int32_t n = iu.n0 + my_dn;
      if (my_m < M && n < iu.nend) {
        const float* b = p.bu[l];
        float v[4] = {z[0], z[1], z[2], z[3]};
        if (b) {
          const float4 bv = *reinterpret_cast<const float4*>(b + n);
          v[0] += bv.x; v[1] += bv.y; v[2] += bv.z; v[3] += bv.w;
        }
        if (p.gated) {
          // gated FFN: H = silu(x W_gate + b_gate) . (x W_up + b_up)
          float g[4] = {zg[0], zg[1], zg[2], zg[3]};
          const float* bgl = p.bg[l];
          if (bgl) {
            const float4 bv = *reinterpret_cast<const float4*>(bgl + n);
            g[0] += bv.x; g[1] += bv.y; g[2] += bv.z; g[3] += bv.w;
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] *= g[e] / (1.0f + __expf(-g[e]));
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = act_apply(p.act, v[e]);
        }
        const uint32_t lo = f32_to_bf16(v[0]) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
        const uint32_t hi = f32_to_bf16(v[2]) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
        if (RES) {
          uint64_t* dst = p.tH + static_cast<int64_t>(my_m) * (p.F / 2) + n / 2;
          st_tagged(dst, lo, static_cast<uint32_t>(l + 1));
          st_tagged(dst + 1, hi, static_cast<uint32_t>(l + 1));
        } else {
          uint32_t* dst = reinterpret_cast<uint32_t*>(p.H + static_cast<int64_t>(my_m) * p.F + n);
          st_agent(dst, lo);
          st_agent(dst + 1, hi);
        }
      }
      if (!RES) {
        wait_vm_all();  // the stores have reached the coherent level
        __syncthreads();
        if (tid == 0) arrive(cnt_up);
      } else {
        __syncthreads();
      }
      // slot 0 is free (every wave passed the barriers above): the next
      // layer's up weights stream in while this workgroup waits
      if (!last) copy(0, p.Wu[l + 1], off_u);
      if (!last && p.gated) copy(2, p.Wg[l + 1], off_u);
    }

    // ---------------- down projection: h += H W_down + b_down ----------------
    if (!RES) wait_for(cnt_up, p.nt_up * (l + 1));
    if (idn.valid && RES) {
      const int s = blockIdx.x % p.ns;
      stage_h(idn, static_cast<uint32_t>(l + 1));
      f32x4_t acc[MB], z;
      compute(1, 1, idn, acc);
      reduce(acc, z);
      const int32_t n = idn.n0 + my_dn;
      const bool mine = my_m < M && n < idn.nend;
      uint64_t* tp = p.tpart + static_cast<int64_t>(l & 1) * p.ns * M * p.D;
      if (mine) {
        uint64_t* dst = tp + (static_cast<int64_t>(s) * M + my_m) * p.D + n;
#pragma unroll
        for (int e = 0; e < 4; ++e) st_tagged(dst + e, __float_as_uint(z[e]), static_cast<uint32_t>(l + 1));
      }
      if (last && s == 0 && mine) {
        // the tile's first chunk sums all of them in chunk order once each
        // carries this layer's tag
        const uint32_t tag = static_cast<uint32_t>(l + 1);
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        for (int c0 = 0; c0 < p.ns; c0 += 4) {
          uint64_t w[16];
          const uint64_t* src[16];
#pragma unroll
          for (int cc = 0; cc < 4; ++cc) {
            const uint64_t* base = tp + (static_cast<int64_t>(min(c0 + cc, p.ns - 1)) * M + my_m) * p.D + n;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              src[4 * cc + e] = c0 + cc < p.ns ? base + e : nullptr;
              w[4 * cc + e] = c0 + cc < p.ns ? ld_tagged(base + e) : 0ull;
            }
          }
          settle_all(src, w, tag, err);
#pragma unroll
          for (int cc = 0; cc < 4; ++cc) {
            if (c0 + cc < p.ns) {
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] += __uint_as_float(static_cast<uint32_t>(w[4 * cc + e]));
            }
          }
        }
        const float* b = p.bd[l];
        if (b) {
          const float4 bv = *reinterpret_cast<const float4*>(b + n);
          v[0] += bv.x; v[1] += bv.y; v[2] += bv.z; v[3] += bv.w;
        }
        const int64_t o = static_cast<int64_t>(my_m) * p.D + n;
        if (p.residual) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += hres[o + e];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) store_out(p.Y, p.ydtype, o + e, v[e]);
      }
      if (!last) copy(1, p.Wd[l + 1], off_d);
    } else if (idn.valid) {
      const int ct = blockIdx.x / p.ns, s = blockIdx.x % p.ns;
      stage_x(idn, p.H, p.F);
      wait_vm_all();
      __syncthreads();
      f32x4_t acc[MB], z;
      compute(1, 1, idn, acc);
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
      {
        if (tid == 0) {
          const int old =
              __hip_atomic_fetch_add(tile_cnt + kCounterStride * ct, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
            if (!last) {
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
          if (tid == 0 && !last) arrive(cnt_dn);
        }
      }
      if (!last) copy(1, p.Wd[l + 1], off_d);
    }
  }
  wait_vm_all();
}

}  // namespace

// Rows per step up to which the running state stays in LDS (RES kernels).
constexpr int kResidentMaxRows = 2;
static_assert(kResidentMaxRows <= 16, "resident kernels cover one 16-row block");
constexpr size_t kStackLdsCap = 150 * 1024;

// slots: up and down weights, plus the gate weights of a gated FFN
static size_t stack_lds_base(int M, int kmax, bool gated) {
  kmax = (kmax + 127) & ~127;
  const size_t xbytes = std::max<size_t>((static_cast<size_t>(M) * kmax * 2 + 1023) & ~size_t(1023), kRedBytes);
  return xbytes + (gated ? 3 : 2) * static_cast<size_t>(kmax / SLICE) * 1024;
}
static size_t stack_lds_res(int M, int kmax, int D, bool gated) {
  const size_t state = (static_cast<size_t>(M) * D * 4 + 1023) & ~size_t(1023);
  return stack_lds_base(M, kmax, gated) + state;
}
// Resident hand-offs keep a down partial buffer per layer parity; a writer
// of layer l + 2 reuses the buffer of layer l once its tile's up items are
// done, which every workgroup's read of layer l precedes only if every
// workgroup owns a down item (each reads all partials before it writes its
// own).
bool decode_stack_resident(int M, int kmax, int D, int ns, bool gated, int nt_up, int nt_dn) {
  return M <= kResidentMaxRows && nt_dn * ns >= nt_up && stack_lds_res(M, kmax, D, gated) <= kStackLdsCap;
}

size_t decode_stack_smem(int M, int kmax, int D, int ns, bool gated) {
  if (M < 1 || M > kDecodeMaxRows || kmax < SLICE || kmax > kMaxSlices * SLICE) return 0;
  const size_t res = stack_lds_res(M, kmax, D, gated);
  const size_t total = M <= kResidentMaxRows && res <= kStackLdsCap ? res : stack_lds_base(M, kmax, gated);
  return total <= kStackLdsCap ? total : 0;
}

template <int MB, bool RES>
static hipError_t launch_stack(const DecodeStack& p, int grid, size_t smem, hipStream_t stream) {
  static std::atomic<unsigned long long> lds_set{0};
  const hipError_t attr =
      ensure_lds_limit(reinterpret_cast<const void*>(decode_stack_kernel<MB, RES>), lds_set, kStackLdsCap);
  if (attr != hipSuccess) return attr;
  DecodeStack arg = p;
  void* args[] = {&arg};
  // An ordinary launch: the grid is at most one workgroup per CU and a
  // workgroup fits on any CU, so on a device that is not held by other work
  // every workgroup is resident at once.  (A cooperative launch, which
  // guarantees that, added about 18 us to every step.)  Should other work hold
  // CUs longer than a wait's bound, the waits time out and the kernel raises
  // its error flag instead of hanging.
  return hipLaunchKernel(reinterpret_cast<const void*>(decode_stack_kernel<MB, RES>), dim3(grid), dim3(kThreads),
                         args, static_cast<unsigned>(smem), stream);
}

hipError_t launch_decode_stack(const DecodeStack& p, int grid, hipStream_t stream) {
  const int kmax = std::max(p.D, p.kc);
  const size_t smem = decode_stack_smem(p.M, kmax, p.D, p.ns, p.gated != 0);
  if (smem == 0) return hipErrorInvalidValue;
  if (decode_stack_resident(p.M, kmax, p.D, p.ns, p.gated != 0, p.nt_up, p.nt_dn)) {
    if (!p.tH || !p.tpart) return hipErrorInvalidValue;
    return launch_stack<1, true>(p, grid, smem, stream);
  }
  switch ((p.M + 15) / 16) {
    case 1: return launch_stack<1, false>(p, grid, smem, stream);
    case 2: return launch_stack<2, false>(p, grid, smem, stream);
    case 3: return launch_stack<3, false>(p, grid, smem, stream);
    default: return launch_stack<4, false>(p, grid, smem, stream);
  }
}

}  // namespace starq
