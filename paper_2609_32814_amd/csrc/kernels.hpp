// Internal host-side interface between the C ABI and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace starq {

constexpr int kMaxQGroups = 64;

enum GemmMode : int { kModeFwd = 0, kModeBwdData = 1, kModeBwdWeight = 2 };

// Arguments of one grouped typed GEMM launch (all three modes).
//
//   FWD        C[rows of type i, output group j] = sum_seg X[rows, seg] W[seg, j]
//   BWD_DATA   C[rows of type i, input group g]  = sum_seg dY[rows, seg] W[g, seg]^T
//   BWD_WEIGHT C[input group g, output group j]  = sum_rows X[rows, g]^T dY[rows, j]
//
// Group starts S (input side of W, K), R (output side of W, N) and the
// column-tile prefix NTp over the column groups of C are host-computed.
struct GemmParams {
  int32_t q;
  int32_t law;  // 0 star, 1 dense, 2 tensor power, 3 graph
  int32_t M;
  int32_t K;
  int32_t N;
  int32_t elem;  // 0 f32, 1 bf16 (operands)
  const int32_t* perm;
  const int32_t* offsets;
  int32_t S[kMaxQGroups + 1];
  int32_t R[kMaxQGroups + 1];
  int32_t NTp[kMaxQGroups + 1];  // column tiles of C per column group, prefix
  int32_t MTp[kMaxQGroups + 1];  // BWD_WEIGHT: row tiles of C per input group, prefix
  const void* A;
  const void* B;
  // FWD epilogue
  const float* bias;
  int32_t act;
  void* Z;
  void* Y;  // FWD: Y; BWD_DATA: dX
  int32_t ydtype;
  // BWD_DATA epilogue
  const void* Zprev;
  // BWD_WEIGHT outputs
  float* dW;
  float* dbias;
  float* partial;     // [nsplit][K][N] when nsplit > 1
  float* dbias_part;  // [nsplit][N] when nsplit > 1
  int32_t nsplit;
  // bf16 pipelined kernel: rows and columns of a C tile (256 x 256, 256 x
  // 192 for the star and dense laws, 192 x 256 for their weight gradient);
  // p.NTp counts column tiles of that width, p.MTp row tiles of that height
  int32_t tile_m, tile_n;
  // law 3 (graph algebra): bit j of adj[i] marks the edge i -> j, bit i of
  // adj_in[j] the same edge (so adj_in[j] holds the in-neighbours of j)
  uint64_t adj[kMaxQGroups];
  uint64_t adj_in[kMaxQGroups];
};

hipError_t launch_type_plan(const int32_t* types, int64_t M, int q, int32_t* perm,
                            int32_t* offsets, hipStream_t stream);
hipError_t launch_count_bad_types(const int32_t* types, int64_t M, int q,
                                  unsigned long long* n_bad, hipStream_t stream);

// Persistent grouped GEMM for fp32 operands: tiles of kTileM rows x 128
// columns (nw must be 2), `grid` workgroups of 256 threads.
hipError_t launch_gemm(int mode, const GemmParams& p, int nw, int grid, hipStream_t stream);
// bf16 forward / activation-gradient / weight-gradient GEMM fed by direct
// global-to-LDS copies: tiles of p.tile_m x p.tile_n (see GemmParams; p.NTp
// and p.MTp must count tiles of that shape); `upper_tiles` bounds
// the tile count and `cus` is the device's CU count (the kernel picks its
// persistent grid from both).
// part[c][n] = sum over rows [c chunk, (c + 1) chunk) of the rows of valid
// type of the bf16 matrix src [M][N]: in row order when every row is valid,
// else in type-sorted order (row perm[position], positions below offsets[q]).
hipError_t launch_column_sum(const uint16_t* src, int32_t N, const int32_t* perm, const int32_t* offsets,
                             int q, int32_t M, int32_t chunk, int nchunks, float* part, hipStream_t stream);
// The same for an fp32 src.
hipError_t launch_column_sum_f32(const float* src, int32_t N, const int32_t* perm, const int32_t* offsets,
                                 int q, int32_t M, int32_t chunk, int nchunks, float* part, hipStream_t stream);
// Law 3 (graph algebra): the output blocks of a forward or activation-gradient
// product that no row's support reaches: for each row of valid type i, the
// columns of every C-column group j that is not a slot of a type-i row
// (forward: output groups j != i with no edge i -> j, written act(bias) and,
// if p.Z, bias; activation gradient: input groups k != i with no edge i -> k,
// written 0).  Every other element of the output is the GEMM's.
hipError_t launch_graph_fill(int mode, const GemmParams& p, hipStream_t stream);
hipError_t launch_gemm_async(int mode, const GemmParams& p, int64_t upper_tiles, int cus,
                             hipStream_t stream);
// Small-tile forward (gemm_narrow.hip): tiles of 64 rows of one type x
// gemm_narrow_cols() columns of one output group; p.NTp counts column tiles
// of that width; n_rb bounds the row blocks over all types.
int gemm_narrow_cols();
int32_t gemm_narrow_row_blocks_upper(int64_t M, int q);
// Its parameters: the forward product for q up to kMaxQFwd groups (the
// star and dense laws; the other laws for q <= kMaxQGroups).
constexpr int kMaxQFwd = 256;
struct NarrowParams {
  int32_t q;
  int32_t law;
  int32_t M;
  int32_t K;
  int32_t N;
  int32_t act;
  int32_t ydtype;
  int32_t swiglu;  // 1: Y is H [M, N / 2] = silu(gate) . up, the N columns gate and up
                   // interleaved in 8-column chunks (Z, if given, the N columns)
  const int32_t* perm;
  const int32_t* offsets;
  const void* A;  // X [M, K] bf16
  const void* B;  // W [K, N] bf16
  const float* bias;
  void* Z;
  void* Y;
  int32_t S[kMaxQFwd + 1];    // input group starts
  int32_t R[kMaxQFwd + 1];    // output group starts
  int32_t NTp[kMaxQFwd + 1];  // column tiles per output group, prefix
  uint64_t adj[kMaxQGroups];  // law 3 (q <= kMaxQGroups): bit j of adj[i] marks the edge i -> j
};
hipError_t launch_gemm_narrow(const NarrowParams& p, int32_t n_rb, int32_t n_ct, int cus, hipStream_t stream);
// Gated FFN elementwise parts (swiglu.hip); n a multiple of 8, elem 1 bf16
// or 0 fp32, 16-byte aligned buffers.
hipError_t launch_swiglu_fwd(int64_t n, int elem, const void* zg, const void* zu, void* h, hipStream_t stream);
// H [M, F] from Z [M, 2F] with gate and up interleaved in 8-feature chunks
hipError_t launch_swiglu_merged(int64_t M, int64_t F, int elem, const void* zgu, void* h, hipStream_t stream);
hipError_t launch_swiglu_bwd(int64_t n, int elem, const void* dh, const void* zg, const void* zu, void* dzg,
                             void* dzu, hipStream_t stream);
hipError_t launch_add(int64_t n, int elem, const void* a, const void* b, void* out, hipStream_t stream);
hipError_t launch_split_reduce(const GemmParams& p, hipStream_t stream);
// out[i] = sum over c < n_parts of part[c * n + i], in c order.
hipError_t launch_sum_partials(const float* part, int n_parts, int64_t n, float* out,
                               hipStream_t stream);
// The same for few outputs (a bias gradient's n columns) over many parts:
// the parts of one output are spread over eight threads, added in a fixed
// order.
hipError_t launch_sum_chunks(const float* part, int nparts, int32_t n, float* out, hipStream_t stream);
// Zero-fills n floats with a kernel (safe to record in a HIP graph).
hipError_t launch_fill_zero(float* dst, int64_t n, hipStream_t stream);

// Rows of C per GEMM tile.
constexpr int kTileM = 256;

// ---- decode ----------------------------------------------------------------

constexpr int kDecodeMaxRows = 64;  // rows per step (one new token per sequence)
constexpr int kDecodeTileN = 16;    // output columns per workgroup
constexpr int kDecodeSliceK = 32;   // K rows per streamed slice
constexpr int kDecodeMaxK = 32768;  // input width of either projection (one-launch-per-projection path)

// One projection of one decode step: out = epilogue(A *_q W + bias) over M
// rows, a workgroup per 16 output columns.
struct DecodePhase {
  int32_t q;
  int32_t law;
  int32_t M;
  int32_t K;  // input width of this projection
  int32_t N;  // output width
  int32_t S[kMaxQGroups + 1];
  int32_t R[kMaxQGroups + 1];
  int32_t NTp[kMaxQGroups + 1];  // column tiles per output group, prefix
  const int32_t* types;
  const uint16_t* A;   // bf16 [M][K]
  const uint16_t* W;   // bf16 [K][N]
  const float* bias;   // [N] or null
  int32_t mode;        // 0: up (out_bf16 = act(z)); 1: down (h = h_prev + z)
  int32_t act;
  int32_t residual;
  uint16_t* out_bf16;     // up: H [M][N]; down: bf16(h) for the next layer, or null
  const float* h_in;      // down, later layers: running state h_prev [M][N] (fp32)
  const uint16_t* h_init; // down, first layer: h_prev read from this bf16 [M][N]
  float* h_out;           // down: new running state [M][N] (fp32), or null
  void* Y;                // down, last layer: final output, or null
  int32_t ydtype;
  uint64_t adj[kMaxQGroups];  // law 3: bit j of adj[i] marks the edge i -> j
  int32_t slots;              // LDS slice slots (set by launch_decode_phase)
};

// The whole decode stack in one persistent launch (see decode_stack.hip).
constexpr int kStackMaxLayers = 32;
struct DecodeStack {
  int32_t q, law, M, D, F, L, act, residual, ydtype;
  int32_t ns, kc;         // down projection: K split into ns chunks of kc
  int32_t nt_up, nt_dn;   // 16-column tiles of F and of D
  int32_t SD[kMaxQGroups + 1];   // D groups: up input, down output
  int32_t SF[kMaxQGroups + 1];   // F groups: up output, down input
  int32_t NTu[kMaxQGroups + 1];  // column-tile prefix over the F groups
  int32_t NTd[kMaxQGroups + 1];  // column-tile prefix over the D groups
  const int32_t* types;
  const uint16_t* X;
  const uint16_t* Wu[kStackMaxLayers];
  const uint16_t* Wd[kStackMaxLayers];
  const float* bu[kStackMaxLayers];
  const float* bd[kStackMaxLayers];
  int32_t gated;                      // gated FFN: H = silu(x W_gate + b_gate) . (x W_up + b_up)
  const uint16_t* Wg[kStackMaxLayers];
  const float* bg[kStackMaxLayers];
  void* Y;
  uint16_t* H;    // [M][F] bf16, the current layer's hidden activation
  uint16_t* hb;   // [2][M][D] bf16, the next up projection's input (layer parity)
  float* h;       // [M][D] fp32 residual state
  float* part;    // [ns][M][D] fp32 down-projection partial sums
  int32_t* cnt;   // decode_stack_counters(nt_dn) int32: (unused) status line, up and down
                  // arrival sub-counters, per-tile down arrivals, each on its own 256-byte line
  int32_t* err;   // error flag: set to 1 when a wait runs out (zero at launch)
  // resident kernels only (zero at launch): 64-bit words (tag << 32 | data),
  // the tag being the layer that wrote the word plus one
  uint64_t* tH;     // [M][F / 2] bf16 pairs of H
  uint64_t* tpart;  // [2][ns][M][D] fp32 down partial sums, by layer parity
  uint64_t adj[kMaxQGroups];  // law 3: bit j of adj[i] marks the edge i -> j
};
// Arrival counters: each sits alone on a 256-byte line (kCounterStride ints).
constexpr int kCounterStride = 64;
constexpr int kSubCounters = 32;
inline int64_t decode_stack_counters(int nt_dn) {
  return static_cast<int64_t>(kCounterStride) * (1 + 2 * kSubCounters + nt_dn);
}
// Dynamic LDS bytes the stack kernel needs, or 0 when the shape does not fit.
size_t decode_stack_smem(int M, int kmax, int D, int ns, bool gated);
// Whether the stack keeps the running state in every workgroup's LDS and hands
// data over as tagged words (then tH and tpart must be set and zero).
bool decode_stack_resident(int M, int kmax, int D, int ns, bool gated, int nt_up, int nt_dn);
// Launches the stack kernel on grid = max(nt_up, nt_dn * ns) <= CU count
// workgroups, which must all be resident at once (an ordinary launch on a
// device not held by other work); p.cnt must be zero.
hipError_t launch_decode_stack(const DecodeStack& p, int grid, hipStream_t stream);

hipError_t launch_decode_phase(DecodePhase p, hipStream_t stream);

// ---- algebraic attention ------------------------------------------------------

// Feature groups of width m = head_dim / q inside every head; layouts are
// token-major: Q and O [B][S][n_heads][head_dim], K and V
// [B][S][n_kv][head_dim] (bf16), query head h reads key/value head
// h / (n_heads / n_kv).
struct AttnParams {
  const void* Q;
  const void* K;
  const void* V;
  void* O;
  int32_t odtype;  // 0 fp32, 1 bf16
  float* lse;      // forward: natural log-sum-exp per (sequence, head, position), or null
  int32_t B, S, n_heads, n_kv, head_dim, q, law;
  // forward: the type plan of the S positions (perm sorted by type, stable)
  const int32_t* perm;
  const int32_t* offsets;
  int32_t items_per_bh;  // grid = B * n_heads * items_per_bh
  // decode: S is the cache capacity; one query row per sequence
  const int32_t* pos_type;   // [S]
  const int32_t* cache_len;  // [B]
  int32_t chunk, nchunks;    // keys per split and splits over S
  int32_t head_groups;       // query heads of one key/value head, in slices of kAttnDecHeads
  float* part_o;             // [B][n_heads][nchunks][head_dim]
  float* part_ml;            // [B][n_heads][nchunks][2]: running max (base 2), sum
};
constexpr int kAttnDecHeads = 8;  // query heads per decode workgroup
constexpr int32_t kAttnFwdMaxSeq = 1 << 18;  // positions per sequence in the forward
// Forward work items per (sequence, head): 128-row query blocks over all types.
inline int32_t attn_fwd_items(int32_t S, int32_t q) { return (S + 127 * q) / 128; }
hipError_t launch_attn_fwd(const AttnParams& p, hipStream_t stream);
// Keys per decode split for a shape (a multiple of the 4 keys per team of
// one batch; the same for every call with that shape).
int32_t attn_decode_chunk(int32_t head_dim, int32_t batch, int32_t n_kv, int32_t head_groups, int32_t S);
hipError_t launch_attn_decode(const AttnParams& p, hipStream_t stream);

// The static workspace of star_decode_noalloc (scratch.hip): its size, and
// its device address on the current device (looked up on the first call per
// device, then cached).
constexpr size_t kDecodeScratchBytes = size_t{4} << 20;
hipError_t decode_scratch(void** ptr);

}  // namespace starq
