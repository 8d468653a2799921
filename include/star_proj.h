/*
 * star_proj.h -- C ABI of the MI355X (gfx950) row-typed associative-algebra
 * projection library (libstarq.so).
 *
 * The operation (Sec. 4, "Transformer Projections", eqs. typed-diag and
 * typed-off; Sec. 5.1, Alg. 1).  X is M x K, W is K x N, both row-major.  The
 * K input features form q contiguous groups of widths s[0..q-1] and the N
 * output features q contiguous groups of widths r[0..q-1]; W_kj is the block
 * of rows of input group k and columns of output group j.  Row b carries a
 * type t_b in [0, q).  A type-i row computes, for every output group j,
 *
 *     y_j = sum over k in B(i,j) of x_k W_kj
 *
 * with B(i,j) = {i, j} as a set for the complete-graph algebra Q_q
 * (STAR_LAW_STAR: y_i = x_i W_ii and y_j = x_i W_ij + x_j W_jj for j != i),
 * or B(i,j) = {0..q-1} for the ordinary product XW (STAR_LAW_DENSE, the
 * same-code dense control).  All q x q blocks of W are parameters; blocks a
 * row's support skips are never read for that row.  The paper's 1-based
 * cyclic schedule tau(p) = 1 + ((p-1) mod q) is t = p mod q for 0-based
 * positions; the library takes the type vector explicitly and bakes in no
 * schedule.
 *
 * Conventions shared by every entry point
 *  - Pointers named "device" are HIP device pointers on the current device;
 *    "host" pointers are read during the call only.  The caller owns and
 *    allocates every buffer, including the workspace; the library keeps no
 *    pointer after a call returns.
 *  - Calls are asynchronous on `stream` (0 = the null stream).  Argument
 *    errors are found on the host before anything is launched: the call then
 *    returns a non-zero status and writes nothing.  A failed launch returns
 *    STAR_ERR_HIP.  Nothing is printed and no exception crosses the ABI.
 *  - Group widths must be positive multiples of 8 and q at most STAR_MAX_Q,
 *    except where an entry point says otherwise: the forward product of the
 *    star and dense laws with bf16 operands (star_proj_fwd,
 *    star_proj_fwd_planned), the type plan and the counting helpers take q
 *    up to STAR_MAX_Q_FWD (the paper's kernel study sweeps q to 256).  A q
 *    in (STAR_MAX_Q, STAR_MAX_Q_FWD] elsewhere is STAR_ERR_UNSUPPORTED; a q
 *    above STAR_MAX_Q_FWD is STAR_ERR_ARG.
 *    Operand, output, bias and workspace pointers must be 16-byte aligned.
 *  - Row types must lie in [0, q).  This is not checked by the compute calls
 *    (star_validate_types checks it).  In the projection and FFN calls a row
 *    with an out-of-range type is left out of every product and its output
 *    row is not written; in the decode calls such a row has an empty support
 *    (see star_decode).  No other row is affected either way.
 *  - M = 0 is a no-op returning STAR_OK.  A type with no rows is legal; the
 *    weight-gradient blocks only that type reaches are written as zeros.
 *  - Operand dtypes: all-F32 or all-BF16 (BF16 operands accumulate in FP32).
 *    Outputs may be F32 or BF16.  Weight and bias gradients are always F32.
 *    Biases are F32.
 *  - Determinism: every output element has one owner and is summed in a fixed
 *    order, so repeated calls on the same inputs give bitwise equal results.
 */
#ifndef STAR_PROJ_H
#define STAR_PROJ_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define STAR_MAX_Q 64
#define STAR_MAX_Q_FWD 256

typedef enum {
    STAR_OK = 0,
    STAR_ERR_ARG = 1,        /* null pointer, bad enum, q out of range */
    STAR_ERR_SHAPE = 2,      /* widths inconsistent, sizes too large */
    STAR_ERR_DTYPE = 3,      /* unsupported dtype combination */
    STAR_ERR_ALIGN = 4,      /* width not a multiple of 8, pointer not 16-byte aligned */
    STAR_ERR_WORKSPACE = 5,  /* workspace missing or smaller than star_workspace_bytes() */
    STAR_ERR_UNSUPPORTED = 6,
    STAR_ERR_HIP = 7         /* a HIP runtime call or launch failed */
} star_status;

typedef enum { STAR_F32 = 0, STAR_BF16 = 1 } star_dtype;

/* Pointwise activation applied after the bias.  GELU is the erf form
 * 0.5 z (1 + erf(z / sqrt 2)); GELU_TANH the tanh approximation.  The paper
 * keeps activations at their usual definitions (Sec. 4, "Projection
 * Shapes").  Every kernel evaluates them in fp32 with the same explicit
 * approximations: values within 1e-6 + 2^-22 |value| of the exact function
 * (the erf form through Abramowitz & Stegun 7.1.28), derivatives within 1e-6
 * (erf form, A&S 7.1.26) or 5e-6 (tanh form). */
typedef enum { STAR_ACT_NONE = 0, STAR_ACT_GELU = 1, STAR_ACT_GELU_TANH = 2 } star_act;

/* STAR_LAW_STAR: B(i,j) = {i,j} (Sec. 5.1).  STAR_LAW_DENSE: all q^2 block
 * products, i.e. the ordinary product XW (eq. dense-two), run through the
 * same kernels as the control.  STAR_LAW_TENSOR2: the tensor power
 * Q_2^{(x)L} of the two-group law (appendix "The Tensor-Square Candidate",
 * eq. recursive-unequal-cost) with q = 2^L groups: a type-i row reaches input
 * group k for output group j when every bit of k equals that bit of i or of
 * j (2^h(i,j) products per output group, 6^L in all).  q must be 1, 2 or 4
 * (STAR_ERR_UNSUPPORTED otherwise); q = 2 is STAR_LAW_STAR, q = 4 the
 * 36-product law of the paper's pretraining pilot.  STAR_LAW_GRAPH: the graph
 * algebra Q_G of a directed graph G without self-loops on the q groups
 * (Sec. "Graph Products with Exact Cost", eqs. graph-basis-products,
 * graph-product-vertex, graph-product-edge): a type-i row's slots are its
 * vertex slot i and the edge slots (i, j) of the edges i -> j, so
 * B(i,i) = {i}, B(i,j) = {i, j} for an edge, and B(i,j) is empty for a
 * non-edge j != i: that output group is not a slot of the row and receives
 * no product (Y = act(bias) there), its input group is never read, and the
 * weight blocks W_ij of non-edges are not parameters (their gradient is
 * written as zeros).  A type-i row costs 1 + 2 outdeg(i) block products,
 * |V| + 2|E| over all types (eq. graph-rank); the complete graph is
 * STAR_LAW_STAR. */
typedef enum { STAR_LAW_STAR = 0, STAR_LAW_DENSE = 1, STAR_LAW_TENSOR2 = 2, STAR_LAW_GRAPH = 3 } star_law;

/* An algebra layout.  s and r are host arrays of q widths (input groups,
 * output groups).  edges: for STAR_LAW_GRAPH a host array of q x q bytes,
 * edges[i * q + j] != 0 for the edge i -> j (the diagonal is ignored), read
 * during the call only; NULL for the other laws (STAR_ERR_ARG if NULL with
 * STAR_LAW_GRAPH). */
typedef struct {
    int32_t q;
    const int64_t *s;
    const int64_t *r;
    star_law law;
    const uint8_t *edges;
} star_algebra;

typedef enum {
    STAR_OP_FWD = 0,
    STAR_OP_BWD_DATA = 1,
    STAR_OP_BWD_WEIGHT = 2,
    STAR_OP_FFN_FWD = 3,
    STAR_OP_DECODE = 4
} star_op;

/*
 * Forward projection with fused bias and activation (Alg. 1; eqs. typed-diag,
 * typed-off): a type-i row's output group j is the sum of x_k W_kj over the
 * input groups k in the law's B(i, j).
 *   row_type  device int32[M]
 *   X         device [M, K] row-major, dtype xt
 *   W         device [K, N] row-major (the canonical bank, never repacked),
 *             dtype wt == xt
 *   bias      device float[N] or NULL; added to every output column for
 *             every row type
 *   Z_out     device [M, N] of dtype yt, or NULL: the pre-activation
 *             Z = X *_q W + bias, kept for the backward pass
 *   Y         device [M, N] of dtype yt: act(Z)
 *   ws        device workspace of at least
 *             star_workspace_bytes(STAR_OP_FWD, alg, NULL, M) bytes
 * q up to STAR_MAX_Q_FWD for the star and dense laws with bf16 operands
 * (the 64 x 128 tiles of star_set_fwd_tiles; STAR_ERR_UNSUPPORTED for other
 * laws or fp32 operands at q > STAR_MAX_Q).
 */
star_status star_proj_fwd(const star_algebra *alg, int64_t M, const int32_t *row_type,
                          const void *X, star_dtype xt, const void *W, star_dtype wt,
                          const float *bias, star_act act, void *Z_out, void *Y,
                          star_dtype yt, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Activation gradient (App. "Vector--Jacobian Products", eqs. vjp-xi and
 * vjp-xj): for a type-i row with output gradient dY,
 *   dX_i = sum_j dY_j W_ij^T   and   dX_k = dY_k W_kk^T (k != i)
 * (law DENSE: dX = dY W^T; in general dX_k = sum of dY_j W_kj^T over the
 * output groups j whose B(i, j) holds k).  If Z_prev is given, the result is multiplied
 * elementwise by act_prev'(Z_prev): the gradient through the activation that
 * produced this projection's input, fused into the epilogue.
 *   dY      device [M, N], dtype dyt
 *   W       device [K, N], dtype wt == dyt
 *   Z_prev  device [M, K] of dtype dyt, or NULL
 *   dX      device [M, K] of dtype dxt, overwritten
 *   ws      at least star_workspace_bytes(STAR_OP_BWD_DATA, alg, NULL, M) bytes
 */
star_status star_proj_bwd_data(const star_algebra *alg, int64_t M, const int32_t *row_type,
                               const void *dY, star_dtype dyt, const void *W, star_dtype wt,
                               const void *Z_prev, star_act act_prev, void *dX,
                               star_dtype dxt, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Weight and bias gradients (eqs. vjp-wii, vjp-wij, vjp-wjj):
 *   dW_jj = sum over all rows of x_j^T dY_j
 *   dW_ij = sum over rows of type i of x_i^T dY_j   (j != i)
 *   dbias = sum over all rows of dY
 * (law DENSE: dW = X^T dY; in general dW_kj sums x_k^T dY_j over the rows whose
 * type i has k in B(i, j)).  dW and dbias are overwritten with the full-batch
 * sums; a block that no row reaches is written as zeros.
 *   X      device [M, K], dtype xt
 *   dY     device [M, N], dtype dyt == xt
 *   dW     device float[K, N]
 *   dbias  device float[N] or NULL
 *   ws     at least star_workspace_bytes(STAR_OP_BWD_WEIGHT, alg, NULL, M) bytes
 */
star_status star_proj_bwd_weight(const star_algebra *alg, int64_t M, const int32_t *row_type,
                                 const void *X, star_dtype xt, const void *dY, star_dtype dyt,
                                 float *dW, float *dbias, void *ws, size_t ws_bytes,
                                 hipStream_t stream);

/*
 * Two-map FFN forward with the same row types on both projections
 * (Sec. 4, "Projection Shapes"; Sec. 5.2):
 *   Z_up = X *_q W_up + b_up;  H = act(Z_up);  Y = H *_q W_down + b_down.
 * up is D -> F, down is F -> D (down's input widths equal up's output
 * widths).  Operands and H have dtype dt; Z_up (optional, for the backward
 * pass) has dtype dt; Y has dtype yt.
 *   X device [M, D]; W_up device [D, F]; W_down device [F, D];
 *   b_up device float[F] or NULL; b_down device float[D] or NULL;
 *   Z_up device [M, F] or NULL; H device [M, F]; Y device [M, D].
 *   ws at least star_workspace_bytes(STAR_OP_FFN_FWD, up, down, M) bytes.
 */
star_status star_ffn_fwd(const star_algebra *up, const star_algebra *down, int64_t M,
                         const int32_t *row_type, const void *X, const void *W_up,
                         const float *b_up, const void *W_down, const float *b_down,
                         star_act act, void *Z_up, void *H, void *Y, star_dtype dt,
                         star_dtype yt, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * One decode step of an FFN stack (Sec. 5.3, "One-Token Inference": the FFN
 * applies Alg. 1 with the new position's row type).  M rows (one new token
 * per sequence, M <= 64) run through n_layers layers of
 *   h <- h + (act(a *_q W_up[l] + b_up[l]) *_q W_down[l] + b_down[l]),
 * where a is h rounded to bfloat16 and h starts as X and is carried in FP32
 * (without `residual` the FFN output replaces h).  The hidden activation is
 * stored in bfloat16.  This is a skinny, weight-bandwidth-bound product: every
 * weight block that some row's support reaches is read once per step, and a
 * block no row's support reaches is not read.  D and F must be at most 32768
 * (STAR_ERR_UNSUPPORTED otherwise); M at most 64.  Shapes whose column tiles
 * fit one workgroup per CU (D, F up to a few thousand) run as one persistent
 * launch for the whole stack; wider ones, and a stack the persistent launch
 * cannot hold, run one launch per projection.  A row whose type lies
 * outside [0, q) reaches no weight block: each layer adds act(b_up) *_q
 * nothing + b_down = b_down, so its Y row is X + the sum of the b_down[l]
 * (without `residual`: b_down of the last layer, or zeros without biases).
 *   row_type  device int32[M]
 *   X         device [M, D] of dtype xt, which must be STAR_BF16 (the
 *             weights are bf16 too); STAR_ERR_DTYPE otherwise
 *   W_up, W_down, b_up, b_down: host arrays of n_layers device pointers
 *             (bf16 [D, F], bf16 [F, D], float[F] or NULL, float[D] or NULL)
 *   Y         device [M, D] of dtype yt: the final h
 *   ws        at least star_workspace_bytes(STAR_OP_DECODE, up, down, M) bytes
 * Where the stack fits, it runs as one persistent launch of at most one
 * workgroup per CU whose workgroups wait on each other, so they must all be
 * resident at once: the device must not be held by long-running work on other
 * streams meanwhile.  If it is, a wait reaches its bound (about half a second),
 * the kernel raises the workspace's error flag, every later wait of the step
 * gives up at once, and the step finishes with an unspecified Y instead of
 * hanging.  star_decode_status reports the flag; every call clears it first.
 */
star_status star_decode(const star_algebra *up, const star_algebra *down, int32_t n_layers,
                        int64_t M, const int32_t *row_type, const void *X, star_dtype xt,
                        const void *const *W_up, const float *const *b_up,
                        const void *const *W_down, const float *const *b_down,
                        star_act act, int32_t residual, void *Y, star_dtype yt,
                        void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * star_decode without a workspace argument and without any allocation, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  The workspace is a
 * static device buffer of STAR_DECODE_SCRATCH_BYTES that the library holds
 * on every device it runs on until the process ends (its address is looked
 * up on the first call on a device); the call itself allocates nothing and
 * frees nothing.  Arguments and results as in star_decode, with these
 * differences:
 *   status  device int32, 4-byte aligned, or NULL: zeroed by the call, then
 *           set to 1 if the step was lost to a wait bound (the flag
 *           star_decode_status reports for star_decode); with NULL the flag
 *           is kept in the static buffer and not reported
 * A shape whose star_decode workspace (star_workspace_bytes(STAR_OP_DECODE,
 * up, down, M)) exceeds STAR_DECODE_SCRATCH_BYTES returns STAR_ERR_WORKSPACE
 * before anything is launched; every shape with D, F <= 4096 and M <= 64
 * fits (wider ones may not).  Every call on one device shares that device's
 * buffer, and each call clears the parts that must start at zero: calls that
 * overlap in time on one device (other streams, other threads) race and
 * give unspecified results; calls ordered on one stream do not.
 */
#define STAR_DECODE_SCRATCH_BYTES (4u << 20)
star_status star_decode_noalloc(const star_algebra *up, const star_algebra *down, int32_t n_layers,
                                int64_t M, const int32_t *row_type, const void *X, star_dtype xt,
                                const void *const *W_up, const float *const *b_up,
                                const void *const *W_down, const float *const *b_down, star_act act,
                                int32_t residual, void *Y, star_dtype yt, int32_t *status,
                                hipStream_t stream);

/*
 * Whether the last star_decode or star_decode_gated call that used workspace
 * `ws` lost its step to a wait bound (see star_decode): waits for the work
 * queued on `stream` (synchronises it), then writes 1 (Y of that call is
 * unspecified) or 0 (no wait ran out) to host *timed_out.
 *   ws  the device workspace passed to that call (the flag is its first
 *       int32); ws_bytes its size, at least 4
 */
star_status star_decode_status(const void *ws, size_t ws_bytes, int32_t *timed_out,
                               hipStream_t stream);

/*
 * star_decode for a gated FFN stack (SwiGLU; Sec. 4, "Projection Shapes", and
 * the pilot's bias-free SwiGLU FFN of Sec. "Small Pretraining Study"):
 *   h <- h + ((silu(a *_q W_gate[l] + b_gate[l]) . (a *_q W_up[l] + b_up[l]))
 *             *_q W_down[l] + b_down[l]),
 * with a, h and H as in star_decode; W_gate has W_up's layout and the same
 * row types.  Runs as the persistent stack only: STAR_ERR_UNSUPPORTED when
 * its three weight slots do not fit in LDS (for D = 768: M above 52).
 *   W_gate, b_gate  host arrays of n_layers device pointers (bf16 [D, F],
 *                   float[F] or NULL); b_gate may be NULL
 *   ws              at least star_workspace_bytes(STAR_OP_DECODE, up, down, M) bytes
 */
star_status star_decode_gated(const star_algebra *up, const star_algebra *down, int32_t n_layers,
                              int64_t M, const int32_t *row_type, const void *X, star_dtype xt,
                              const void *const *W_gate, const float *const *b_gate,
                              const void *const *W_up, const float *const *b_up,
                              const void *const *W_down, const float *const *b_down,
                              int32_t residual, void *Y, star_dtype yt, void *ws, size_t ws_bytes,
                              hipStream_t stream);

/*
 * Type plan: the per-type row sets I_i of Algorithm alg:projection (the rows
 * whose position has type i) as one stable permutation of the rows grouped
 * by type plus q+1 offsets.  Every compute call needs it; the plain entry points build it in
 * their workspace on each call, the *_planned entry points take one built
 * here, so calls that share row types (the six products of an FFN training
 * step, repeated replays) build it once.
 *   plan  device buffer of at least star_plan_bytes(q, M) bytes, 16-byte
 *         aligned; it holds int32 perm[M] followed (at a 256-byte boundary)
 *         by int32 offsets[q+1].  Rows with a type outside [0, q) are placed
 *         after offsets[q] and left out of every product.
 */
 /* q up to STAR_MAX_Q_FWD. */
size_t star_plan_bytes(int32_t q, int64_t M);
star_status star_type_plan(int32_t q, int64_t M, const int32_t *row_type, void *plan,
                           size_t plan_bytes, hipStream_t stream);

/* star_proj_fwd with a plan built by star_type_plan for the same rows (no
 * workspace needed). */
star_status star_proj_fwd_planned(const star_algebra *alg, int64_t M, const void *plan,
                                  const void *X, star_dtype xt, const void *W, star_dtype wt,
                                  const float *bias, star_act act, void *Z_out, void *Y,
                                  star_dtype yt, hipStream_t stream);

/* star_proj_bwd_data with a prebuilt plan (no workspace needed). */
star_status star_proj_bwd_data_planned(const star_algebra *alg, int64_t M, const void *plan,
                                       const void *dY, star_dtype dyt, const void *W,
                                       star_dtype wt, const void *Z_prev, star_act act_prev,
                                       void *dX, star_dtype dxt, hipStream_t stream);

/* star_proj_bwd_weight with a prebuilt plan.  ws holds the split partial
 * sums: at least star_workspace_bytes(STAR_OP_BWD_WEIGHT, alg, NULL, M)
 * bytes (may be NULL when that size equals star_plan_bytes(q, M)). */
star_status star_proj_bwd_weight_planned(const star_algebra *alg, int64_t M, const void *plan,
                                         const void *X, star_dtype xt, const void *dY,
                                         star_dtype dyt, float *dW, float *dbias, void *ws,
                                         size_t ws_bytes, hipStream_t stream);

/* Tile size of the forward product for bf16 operands (Sec. "Kernel Scaling
 * on Transformer Shapes": the algebraic kernel's tile is calibrated per
 * shape).  STAR_TILES_AUTO, the default, takes tiles of 64 rows x 128
 * columns when the 256 x 256 tiles would be at most three quarters full
 * (rows taken as spread evenly over the types) and a tile contracts over
 * fewer than 1024 input features on average (K for the dense law, two
 * groups' worth otherwise), or when they would be fewer than 128; else
 * tiles of 256 rows x 256 columns, or x 192 columns (star and dense laws)
 * where those pad fewer output columns (groups 384 wide) and an estimate of
 * the persistent kernel's tile deal favours them.  STAR_TILES_WIDE (256 x
 * 256), STAR_TILES_WIDE192 (256 x 192 for the star and dense laws, 256 x
 * 256 for the others) and STAR_TILES_SMALL force one size.  Input groups
 * narrower than 64 always take the small tiles, fp32 operands always their
 * own kernel.  Applies to star_proj_fwd, star_proj_fwd_planned and the
 * projections of star_ffn_fwd.  Process-wide (every device and stream),
 * read when a call launches.  Returns the previous choice, or -1 (nothing
 * changed) for a value outside the enum.  Both sizes give the same results
 * to rounding: the K order within a group is the same, the tiles differ. */
typedef enum {
  STAR_TILES_AUTO = 0,
  STAR_TILES_WIDE = 1,
  STAR_TILES_SMALL = 2,
  STAR_TILES_WIDE192 = 3
} star_tiles;
int star_set_fwd_tiles(int tiles);

/* Workspace bytes an entry point needs (alg2 is the down algebra for
 * STAR_OP_FFN_FWD and STAR_OP_DECODE, else ignored).  Returns 0 for invalid
 * arguments. */
size_t star_workspace_bytes(int32_t op, const star_algebra *alg, const star_algebra *alg2,
                            int64_t M);

/* Block products a type-i row evaluates, written to host per_type[q]:
 * 2q-1 for STAR_LAW_STAR (eq. q-rank: 2q^2 - q over all types), q^2 for
 * STAR_LAW_DENSE. */
star_status star_count_products(const star_algebra *alg, int64_t *per_type);

/* Multiply-accumulates of one forward pass over rows with the given
 * per-type counts (eq. rectangular-batch-cost):
 * sum_i rows_per_type[i] * (D_diag + s_i (N - r_i)) for the star law. */
star_status star_count_macs(const star_algebra *alg, const int64_t *rows_per_type,
                            int64_t *macs);

/* Counts the rows whose type lies outside [0, q) and stores the count in
 * host *n_bad.  Synchronises `stream`.  ws: at least 16 bytes of device
 * memory. */
star_status star_validate_types(int64_t M, const int32_t *row_type, int32_t q,
                                int64_t *n_bad, void *ws, size_t ws_bytes,
                                hipStream_t stream);

/*
 * Gated FFN (SwiGLU) pieces.  The paper's gated FFN has two D x F maps (gate
 * and up) and one F x D map, each a row-typed projection with the same row
 * types (Sec. 4, "Projection Shapes"; Sec. "Small Pretraining Study", the pilot's
 * bias-free SwiGLU FFN); the gate and the product keep their usual
 * definitions.  The three projections run through star_proj_*; these calls
 * are the elementwise steps between them.  n elements (a multiple of 8) of
 * dtype dt, every buffer device memory, 16-byte aligned, not overlapping;
 * silu(z) = z / (1 + exp(-z)).
 *   star_swiglu_fwd:  H = silu(Z_gate) . Z_up
 *   star_swiglu_bwd:  dZ_gate = dH . Z_up . silu'(Z_gate);  dZ_up = dH . silu(Z_gate)
 *   star_add:         out = a + b (the two activation gradients of a gated
 *                     FFN's input); out may alias a or b.
 */
star_status star_swiglu_fwd(int64_t n, const void *Z_gate, const void *Z_up, star_dtype dt, void *H,
                            hipStream_t stream);
star_status star_swiglu_bwd(int64_t n, const void *dH, const void *Z_gate, const void *Z_up,
                            star_dtype dt, void *dZ_gate, void *dZ_up, hipStream_t stream);
star_status star_add(int64_t n, const void *a, const void *b, star_dtype dt, void *out,
                     hipStream_t stream);

/*
 * Merged gate/up (§"Kernel Benchmark Details": the SwiGLU comparison merges
 * the gate and up projections on both sides; Tab. kernel-ffn).  The two
 * D x F maps share the row types and the input, so they run as one D x 2F
 * product whose output columns hold gate and up interleaved in 8-feature
 * chunks: feature f's gate at column 16 (f / 8) + f % 8, its up value 8
 * columns on.  With the output groups of the up layout r_j (multiples of 8),
 * the merged algebra has output widths 2 r_j and the same law; its weight
 * bank W_gu [D, 2F] and bias b_gu [2F] are W_gate, W_up (and b_gate, b_up)
 * interleaved the same way.
 *   star_swiglu_merged_fwd: H [M, F] = silu(gate) . up from the merged
 *       product's output Z_gu [M, 2F] (dtype dt; F a multiple of 8; every
 *       buffer device memory, 16-byte aligned).
 *   star_swiglu_up_fwd_planned: the merged product with SwiGLU applied in
 *       its epilogue: H [M, F] (dtype ht) = silu(Z_gate) . Z_up, Z from the
 *       fp32 accumulators (plus b_gu if given), never stored unless Z_out
 *       (the merged pre-activation [M, 2F], dtype ht) is given.  bf16 X and
 *       W_gu; plan from star_type_plan; q up to STAR_MAX_Q_FWD; the star,
 *       dense and tensor laws (STAR_ERR_UNSUPPORTED for the graph law or an
 *       output width not a multiple of 16).
 */
star_status star_swiglu_merged_fwd(int64_t M, int64_t F, const void *Z_gu, star_dtype dt, void *H,
                                   hipStream_t stream);
star_status star_swiglu_up_fwd_planned(const star_algebra *alg_gu, int64_t M, const void *plan,
                                       const void *X, star_dtype xt, const void *W_gu, star_dtype wt,
                                       const float *b_gu, void *Z_out, void *H, star_dtype ht,
                                       hipStream_t stream);

/*
 * Algebraic attention (appendix "Attention Extension and Detailed Cost
 * Accounting"; Algs. attention-training and attention-decoding, their score
 * and aggregation steps).  Each head of width d_h = q m is split into q
 * feature groups of width m.  For a query at position p of type i and a key
 * at position u <= p of type j, the score keeps the groups a in F(i, j):
 *
 *     s_pu = sum over a in F(i, j) of <Q_p^(a), K_u^(a)> / sqrt(|F(i, j)| m)
 *
 * (eqs. feature-set, attention-raw-score, attention-support-size,
 * attention-score), with F(i, i) = {i}, F(i, j) = {i, j} for STAR_LAW_STAR,
 * every group for STAR_LAW_DENSE (ordinary attention with the 1/sqrt(d_h)
 * rule: the same-code control), and the groups whose every bit equals that
 * bit of i or of j for STAR_LAW_TENSOR2 (eq. tensor-square-feature-set,
 * q = 1, 2 or 4).  Keys after the query are masked (eq. causal-mask); the
 * output is the softmax-weighted sum of the full value rows (eq. softmax-pv).
 * Softmax and accumulation run in fp32; the probabilities enter the value
 * product rounded to bf16.
 *
 * Layouts (row-major, token-major): Q and O hold [batch][seq_len][n_heads]
 * [head_dim], K and V [batch][seq_len][n_kv_heads][head_dim]; query head h
 * uses key/value head h / (n_heads / n_kv_heads) (grouped-query attention).
 * Group a of a head is its features [a m, (a + 1) m).  Q, K and V are BF16,
 * O is F32 or BF16; every tensor pointer 16-byte aligned.  STAR_LAW_GRAPH is
 * not defined for attention (STAR_ERR_UNSUPPORTED).
 */
typedef struct {
    int32_t batch;       /* sequences B (0: no-op) */
    int32_t seq_len;     /* forward: positions S per sequence; decode: cache capacity */
    int32_t n_heads;     /* query heads */
    int32_t n_kv_heads;  /* key/value heads, dividing n_heads */
    int32_t head_dim;    /* d_h: 64 or 128 (STAR_ERR_UNSUPPORTED otherwise) */
    int32_t q;           /* groups per head; m = head_dim / q a multiple of 8 */
    star_law law;
} star_attn_shape;

/* Causal forward over whole sequences (training or prefill).
 *   plan  device plan of the position types, built by
 *         star_type_plan(q, seq_len, pos_type, ...) from device
 *         int32 pos_type[seq_len], the type of each position (the same for
 *         every sequence).  A position whose type lies outside [0, q) is
 *         neither a query nor a key and its output rows are not written.
 *   lse   device float[batch][n_heads][seq_len] or NULL: the natural
 *         log-sum-exp of each query's scaled scores (the softmax
 *         normaliser a backward pass needs).
 * Errors: STAR_ERR_ARG (null pointer, bad law), STAR_ERR_SHAPE (a size
 * below zero, n_kv_heads not dividing n_heads, seq_len above 262144, a grid
 * too large),
 * STAR_ERR_UNSUPPORTED (head_dim, q or m outside the supported set),
 * STAR_ERR_DTYPE, STAR_ERR_ALIGN. */
star_status star_attn_fwd(const star_attn_shape *shape, const void *plan, const void *Q,
                          const void *K, const void *V, star_dtype dt, void *O, star_dtype ot,
                          float *lse, hipStream_t stream);

/* One decode step over a KV cache (Alg. attention-decoding): one new query
 * row per sequence, attending to the cached keys and values at positions
 * 0 .. cache_len[b] - 1, the last of which is the query's own position (its
 * key and value already appended by the caller).  The cache keeps every
 * feature of every key (eq. kv-cache-shape): a later query of another type
 * reads other groups of the same key.
 *   shape->seq_len  the cache capacity S_max
 *   pos_type   device int32[S_max]: the type of each cache position
 *   cache_len  device int32[batch]: valid cache entries per sequence; values
 *              above S_max count as S_max; a sequence with cache_len <= 0,
 *              or whose query position has a type outside [0, q), gets a zero
 *              output row.  Cached keys of a type outside [0, q) are skipped.
 *   Q          device [batch][n_heads][head_dim], BF16
 *   K_cache, V_cache  device [batch][S_max][n_kv_heads][head_dim], BF16
 *   O          device [batch][n_heads][head_dim] of dtype ot
 *   ws         device workspace of star_attn_decode_workspace_bytes(shape)
 *              bytes: the per-chunk partial results.
 * The cache is split into chunks of 128 (head_dim 64) or 64 (head_dim 128)
 * positions, each read once for the up to 8 query heads of one key/value
 * head that one workgroup serves; a second kernel merges the chunks. */
size_t star_attn_decode_workspace_bytes(const star_attn_shape *shape);
star_status star_attn_decode(const star_attn_shape *shape, const int32_t *pos_type,
                             const int32_t *cache_len, const void *Q, const void *K_cache,
                             const void *V_cache, star_dtype dt, void *O, star_dtype ot, void *ws,
                             size_t ws_bytes, hipStream_t stream);

/* Static description of a status code. */
const char *star_status_string(star_status s);

#ifdef __cplusplus
}
#endif

#endif /* STAR_PROJ_H */
