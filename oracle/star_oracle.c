/*
 * star_oracle.c -- plain fp64 CPU oracle for the row-typed associative-algebra
 * projection Y = X *_q W ("Change the Product, Keep the Parameters:
 * Associative Algebra Layers for Transformers").
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or helper with the HIP
 * path.
 *
 * Every routine is the plain definition written out in fp64: no blocking, no
 * fusion, no BLAS.  Loops run over rows (OpenMP), then over the algebra's
 * support, then over the scalars of each block product.
 *
 * Notation (Sec. 4, "Transformer Projections"):
 *   X in F^{M x K}, W in F^{K x N}, both row-major and dense.
 *   Input features split into q contiguous groups of widths s_0..s_{q-1}
 *   (K = sum s), output features into q contiguous groups of widths
 *   r_0..r_{q-1} (N = sum r).  Block W_{kj} is rows [S_k, S_k+s_k) and
 *   columns [R_j, R_j+r_j) of W, with S, R the exclusive prefix sums.
 *   Row b carries a type t_b in {0..q-1}; the paper's 1-based type
 *   tau(p) = 1 + ((p-1) mod q) is t = p0 mod q with 0-based positions p0.
 *
 * Support B(i,j) (Sec. 5.1, eq. recursive-row-action): the set of input
 * groups k whose block product x_k W_{kj} a type-i row accumulates into its
 * output group j.
 *   law 0 (complete-graph algebra Q_q): B(i,j) = {i, j} as a set, so the
 *          diagonal product x_i W_ii is counted once (eqs. typed-diag,
 *          typed-off).
 *   law 1 (ordinary product, the dense control): B(i,j) = {0..q-1}
 *          (eq. dense-two for q = 2).
 *   law 2 (tensor power Q_2^{(x)L} of the two-group law, q = 2^L; appendix
 *          "The Tensor-Square Candidate", eq. recursive-unequal-cost): types
 *          and group indices are bit strings of length L (index
 *          g = sum_k g_k 2^k), and a type-a row reaches input group b for
 *          output group d when every bit of b equals the same bit of a or of
 *          d.  L = 1 is Q_2; L = 2 is the pilot's 36-product law.
 *   law 3 (graph algebra Q_G of a directed graph G on the q groups without
 *          self-loops; Sec. "Graph Products with Exact Cost", eqs.
 *          graph-basis-products, graph-product-vertex, graph-product-edge):
 *          the slots of a type-i row are its vertex slot i and the edge slots
 *          (i, j) of the edges leaving i.  So B(i,i) = {i}; B(i,j) = {i, j}
 *          for an edge i -> j; and B(i,j) is empty for a non-edge j != i: that
 *          output group is not a slot of the row, its product is zero (the
 *          bias and activation still apply, as everywhere).  edges[i q + j]
 *          != 0 marks the edge i -> j (the diagonal is ignored).  The
 *          complete graph is law 0.
 *
 * Every routine that takes a law also takes `edges` (q x q bytes, read for
 * law 3 only; NULL otherwise).
 *
 * Activations: 0 none, 1 GELU with the exact erf form
 * 0.5 z (1 + erf(z / sqrt 2)), 2 GELU with the tanh form, 3 SiLU
 * z / (1 + exp(-z)) (the gate of a SwiGLU FFN).  The paper keeps
 * biases and pointwise activations at their usual definitions (Sec. 4,
 * "Projection Shapes"); which activation to use is not fixed by the paper.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_LAW_STAR 0
#define ORACLE_LAW_DENSE 1
#define ORACLE_LAW_TENSOR2 2
#define ORACLE_LAW_GRAPH 3

#define ORACLE_ACT_NONE 0
#define ORACLE_ACT_GELU 1
#define ORACLE_ACT_GELU_TANH 2
#define ORACLE_ACT_SILU 3

/* k in B(i,j)?  Sec. 5.1: B(i,j) = {i,j} as a set for Q_q; all k for the
 * ordinary product. */
int oracle_in_support(int law, const unsigned char *edges, int q, int i, int j, int k)
{
    if (law == ORACLE_LAW_DENSE) return 1;
    if (law == ORACLE_LAW_GRAPH) {
        if (j == i) return k == i;
        if (!edges || !edges[i * q + j]) return 0; /* output group j is no slot of a type-i row */
        return k == i || k == j;                   /* x_i W_ij + x_j W_jj */
    }
    if (law == ORACLE_LAW_TENSOR2) {
        /* beta_k in {alpha_k, delta_k} for every bit k */
        for (int bit = 0; bit < 30; ++bit) {
            const int b = (k >> bit) & 1, a = (i >> bit) & 1, d = (j >> bit) & 1;
            if (b != a && b != d) return 0;
        }
        return 1;
    }
    return k == i || k == j;
}

static void prefix(int q, const int64_t *w, int64_t *P)
{
    P[0] = 0;
    for (int g = 0; g < q; ++g) P[g + 1] = P[g] + w[g];
}

/* ---- activations -------------------------------------------------------- */

static const double kSqrt2 = 1.41421356237309504880;
static const double kSqrt2OverPi = 0.79788456080286535588;  /* sqrt(2/pi) */
static const double kInvSqrt2Pi = 0.39894228040143267794;   /* 1/sqrt(2 pi) */

double oracle_act(int act, double z)
{
    switch (act) {
    case ORACLE_ACT_GELU:
        return 0.5 * z * (1.0 + erf(z / kSqrt2));
    case ORACLE_ACT_GELU_TANH: {
        double u = kSqrt2OverPi * (z + 0.044715 * z * z * z);
        return 0.5 * z * (1.0 + tanh(u));
    }
    case ORACLE_ACT_SILU:
        return z / (1.0 + exp(-z));
    default:
        return z;
    }
}

/* d act / dz.  Exact GELU: Phi(z) + z phi(z).  Tanh GELU: derivative of
 * 0.5 z (1 + tanh(u(z))) with u = sqrt(2/pi) (z + 0.044715 z^3). */
double oracle_act_grad(int act, double z)
{
    switch (act) {
    case ORACLE_ACT_GELU:
        return 0.5 * (1.0 + erf(z / kSqrt2)) + z * kInvSqrt2Pi * exp(-0.5 * z * z);
    case ORACLE_ACT_GELU_TANH: {
        double u = kSqrt2OverPi * (z + 0.044715 * z * z * z);
        double t = tanh(u);
        double du = kSqrt2OverPi * (1.0 + 3.0 * 0.044715 * z * z);
        return 0.5 * (1.0 + t) + 0.5 * z * (1.0 - t * t) * du;
    }
    case ORACLE_ACT_SILU: {
        /* s + z s (1 - s) with s the logistic sigmoid */
        double sg = 1.0 / (1.0 + exp(-z));
        return sg + z * sg * (1.0 - sg);
    }
    default:
        return 1.0;
    }
}

/* Round a double to the nearest bfloat16 value (8 significant bits, ties to
 * even, binary32 exponent range), returned as a double.  Used to mirror the
 * tensors that the GPU path stores in bfloat16 between two products. */
double oracle_round_bf16(double x)
{
    if (isnan(x) || isinf(x) || x == 0.0) return x;
    double ax = fabs(x);
    /* largest finite bf16: (2 - 2^-7) * 2^127; halfway to 2^128 overflows */
    const double maxbf = ldexp(255.0, 120);
    const double halfway = ldexp(511.0, 119);
    if (ax >= halfway) return x > 0 ? INFINITY : -INFINITY;
    int e;
    frexp(ax, &e);            /* ax = m 2^e, m in [0.5, 1) */
    int ulp_exp = e - 8;      /* 8 significant bits */
    if (ulp_exp < -133) ulp_exp = -133; /* bf16 subnormal quantum 2^-133 */
    double scaled = ldexp(ax, -ulp_exp);
    double r = nearbyint(scaled);     /* default rounding: ties to even */
    double y = ldexp(r, ulp_exp);
    if (y > maxbf) y = maxbf;
    return x < 0 ? -y : y;
}

void oracle_round_bf16_array(int64_t n, const double *x, double *y)
{
    for (int64_t i = 0; i < n; ++i) y[i] = oracle_round_bf16(x[i]);
}

/* ---- product counts (Prop. "Parameters and Rectangular Cost") ------------ */

/* Number of block products a type-i row visits in Alg. 1: the pairs (j,k)
 * with k in B(i,j).  2q-1 for Q_q (eq. q-rank counts 2q^2 - q over all q
 * types), q^2 for the ordinary product. */
int64_t oracle_products_per_type(int law, const unsigned char *edges, int q, int i)
{
    int64_t n = 0;
    for (int j = 0; j < q; ++j)
        for (int k = 0; k < q; ++k)
            n += oracle_in_support(law, edges, q, i, j, k);
    return n;
}

/* MACs of one type-i row: sum over visited (j,k) of s_k r_j
 * (eq. unequal-row-cost for Q_q: C_i = D_diag + s_i (N - r_i)). */
int64_t oracle_row_macs(int law, const unsigned char *edges, int q, const int64_t *s, const int64_t *r, int i)
{
    int64_t n = 0;
    for (int j = 0; j < q; ++j)
        for (int k = 0; k < q; ++k)
            if (oracle_in_support(law, edges, q, i, j, k)) n += s[k] * r[j];
    return n;
}

/* ---- forward: Alg. 1 ----------------------------------------------------- */

/*
 * Alg. 1 (batched or one-token projection), followed by the usual bias and
 * pointwise activation:
 *   Y <- 0
 *   for each row type i:
 *     I_i <- {b : t_b = i}
 *     for each output group j and each k in B(i,j):
 *       Y_j[I_i] <- Y_j[I_i] + X_k[I_i] W_kj
 *   Z = Y + bias (every output column, every row type);  out = act(Z)
 *
 * Z_out (pre-activation) may be NULL.  Returns the number of MACs visited
 * (sum over rows of C_{t_b}); products_per_type[i] (may be NULL) receives the
 * number of block products a type-i row visits.  Returns -1 on an
 * out-of-range type.
 */
int64_t oracle_proj_fwd(int q, const int64_t *s, const int64_t *r, int law, const unsigned char *edges,
                        int64_t M, const int32_t *t,
                        const double *X, const double *W, const double *bias,
                        int act, double *Z_out, double *Y,
                        int64_t *products_per_type)
{
    int64_t *S = malloc(sizeof(int64_t) * (q + 1));
    int64_t *R = malloc(sizeof(int64_t) * (q + 1));
    prefix(q, s, S);
    prefix(q, r, R);
    const int64_t K = S[q], N = R[q];
    for (int64_t b = 0; b < M; ++b)
        if (t[b] < 0 || t[b] >= q) { free(S); free(R); return -1; }

    memset(Y, 0, sizeof(double) * (size_t)(M * N));
    int64_t macs = 0;
    int64_t *I = malloc(sizeof(int64_t) * (M > 0 ? M : 1));
    for (int i = 0; i < q; ++i) {
        int64_t Mi = 0;
        for (int64_t b = 0; b < M; ++b)
            if (t[b] == i) I[Mi++] = b;                 /* I_i */
        if (products_per_type) products_per_type[i] = oracle_products_per_type(law, edges, q, i);
        for (int j = 0; j < q; ++j) {
            for (int k = 0; k < q; ++k) {
                if (!oracle_in_support(law, edges, q, i, j, k)) continue;
                /* Y_j[I_i] += X_k[I_i] W_kj */
                #pragma omp parallel for schedule(static)
                for (int64_t m = 0; m < Mi; ++m) {
                    const int64_t b = I[m];
                    const double *xk = X + b * K + S[k];
                    double *yj = Y + b * N + R[j];
                    for (int64_t e = 0; e < s[k]; ++e) {
                        const double xe = xk[e];
                        const double *wrow = W + (S[k] + e) * N + R[j];
                        for (int64_t c = 0; c < r[j]; ++c) yj[c] += xe * wrow[c];
                    }
                }
                macs += Mi * s[k] * r[j];
            }
        }
    }
    free(I);
    #pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < M; ++b) {
        for (int64_t n = 0; n < N; ++n) {
            double z = Y[b * N + n] + (bias ? bias[n] : 0.0);
            if (Z_out) Z_out[b * N + n] = z;
            Y[b * N + n] = oracle_act(act, z);
        }
    }
    free(S);
    free(R);
    return macs;
}

/* ---- backward (App. "Vector--Jacobian Products") ------------------------- */

/*
 * Activation gradient.  For a type-i row with output gradient ybar, the VJPs
 * (eqs. vjp-xi, vjp-xj) are
 *   xbar_i += ybar_i W_ii^T + sum_{j != i} ybar_j W_ij^T
 *   xbar_j += ybar_j W_jj^T                      (j != i)
 * i.e. xbar_k += ybar_j W_kj^T for every (j, k) with k in B(i,j); the same
 * support rule covers the ordinary product.  If Zprev is given, the result is
 * multiplied elementwise by act'(Zprev) (the gradient through the activation
 * that produced this projection's input).  dX is overwritten.
 */
int oracle_proj_bwd_data(int q, const int64_t *s, const int64_t *r, int law, const unsigned char *edges,
                         int64_t M, const int32_t *t,
                         const double *dY, const double *W,
                         const double *Zprev, int act_prev, double *dX)
{
    int64_t S[q + 1], R[q + 1];
    prefix(q, s, S);
    prefix(q, r, R);
    const int64_t K = S[q], N = R[q];
    for (int64_t b = 0; b < M; ++b)
        if (t[b] < 0 || t[b] >= q) return -1;
    #pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < M; ++b) {
        const int i = t[b];
        double *xb = dX + b * K;
        for (int64_t c = 0; c < K; ++c) xb[c] = 0.0;
        for (int j = 0; j < q; ++j) {
            const double *yj = dY + b * N + R[j];
            for (int k = 0; k < q; ++k) {
                if (!oracle_in_support(law, edges, q, i, j, k)) continue;
                double *xk = xb + S[k];
                for (int64_t e = 0; e < s[k]; ++e) {
                    const double *wrow = W + (S[k] + e) * N + R[j];
                    double acc = 0.0;
                    for (int64_t c = 0; c < r[j]; ++c) acc += yj[c] * wrow[c];
                    xk[e] += acc;
                }
            }
        }
        if (Zprev)
            for (int64_t c = 0; c < K; ++c)
                xb[c] *= oracle_act_grad(act_prev, Zprev[b * K + c]);
    }
    return 0;
}

/*
 * Weight and bias gradients (eqs. vjp-wii, vjp-wij, vjp-wjj): for each row b
 * of type i and each (j, k) with k in B(i,j),  Wbar_kj += x_k^T ybar_j;
 * dbias = sum_b ybar_b.  Both are overwritten with the full-batch sum, so a
 * block that no row's support reaches comes out zero.
 */
int oracle_proj_bwd_weight(int q, const int64_t *s, const int64_t *r, int law, const unsigned char *edges,
                           int64_t M, const int32_t *t,
                           const double *X, const double *dY,
                           double *dW, double *dbias)
{
    int64_t S[q + 1], R[q + 1];
    prefix(q, s, S);
    prefix(q, r, R);
    const int64_t K = S[q], N = R[q];
    for (int64_t b = 0; b < M; ++b)
        if (t[b] < 0 || t[b] >= q) return -1;
    memset(dW, 0, sizeof(double) * (size_t)(K * N));
    /* parallel over the rows of dW (input features): each thread owns whole
     * rows of dW, then walks the batch in order */
    #pragma omp parallel for schedule(static)
    for (int64_t kk = 0; kk < K; ++kk) {
        int k = 0;
        while (kk >= S[k + 1]) ++k;
        double *dwrow = dW + kk * N;
        for (int64_t b = 0; b < M; ++b) {
            const int i = t[b];
            const double xe = X[b * K + kk];
            for (int j = 0; j < q; ++j) {
                if (!oracle_in_support(law, edges, q, i, j, k)) continue;
                const double *yj = dY + b * N + R[j];
                double *dwj = dwrow + R[j];
                for (int64_t c = 0; c < r[j]; ++c) dwj[c] += xe * yj[c];
            }
        }
    }
    if (dbias) {
        for (int64_t n = 0; n < N; ++n) dbias[n] = 0.0;
        for (int64_t b = 0; b < M; ++b)
            for (int64_t n = 0; n < N; ++n) dbias[n] += dY[b * N + n];
    }
    return 0;
}

/* ---- square block arrays (Sec. 3.2, eqs. q-product-diag/-off) ----------- */

/*
 * C = A *_q B for square block arrays with q x q blocks of size b x b
 * (side n = q b, row-major):
 *   (A*B)_ii = A_ii B_ii
 *   (A*B)_ij = A_ii B_ij + A_ij B_jj   (i != j)
 * Written directly from the square rule, independently of the typed
 * projection above.
 */
void oracle_square_law(int law, const unsigned char *edges, int q, int64_t bs, const double *A, const double *B, double *C);

void oracle_square_star(int q, int64_t bs, const double *A, const double *B, double *C)
{
    const int64_t n = q * bs;
    memset(C, 0, sizeof(double) * (size_t)(n * n));
    #define BLK(P, i, j, u, v) (P)[((i) * bs + (u)) * n + (j) * bs + (v)]
    for (int i = 0; i < q; ++i)
        for (int j = 0; j < q; ++j)
            for (int64_t u = 0; u < bs; ++u)
                for (int64_t v = 0; v < bs; ++v) {
                    double acc = 0.0;
                    for (int64_t w = 0; w < bs; ++w) {
                        acc += BLK(A, i, i, u, w) * BLK(B, i, j, w, v);
                        if (i != j) acc += BLK(A, i, j, u, w) * BLK(B, j, j, w, v);
                    }
                    BLK(C, i, j, u, v) = acc;
                }
    #undef BLK
}

/*
 * Selected entries of the weight gradient, one by one:
 *   dW[kk][n] = sum over rows b with k in B(t_b, j) of X[b][kk] dY[b][n],
 * where k is the input group of kk and j the output group of n
 * (eqs. vjp-wii, vjp-wij, vjp-wjj).  For checking large shapes, where the
 * full gradient is too slow to form on the CPU.
 */
int oracle_bwd_weight_entries(int q, const int64_t *s, const int64_t *r, int law, const unsigned char *edges,
                              int64_t M, const int32_t *t,
                              const double *X, const double *dY,
                              int64_t n_entries, const int64_t *kk_idx,
                              const int64_t *n_idx, double *out)
{
    int64_t S[q + 1], R[q + 1];
    prefix(q, s, S);
    prefix(q, r, R);
    const int64_t K = S[q], N = R[q];
    for (int64_t b = 0; b < M; ++b)
        if (t[b] < 0 || t[b] >= q) return -1;
    #pragma omp parallel for schedule(dynamic, 16)
    for (int64_t e = 0; e < n_entries; ++e) {
        const int64_t kk = kk_idx[e], n = n_idx[e];
        int k = 0, j = 0;
        while (kk >= S[k + 1]) ++k;
        while (n >= R[j + 1]) ++j;
        double acc = 0.0;
        for (int64_t b = 0; b < M; ++b)
            if (oracle_in_support(law, edges, q, t[b], j, k)) acc += X[b * K + kk] * dY[b * N + n];
        out[e] = acc;
    }
    return 0;
}

/* Number of OpenMP threads the parallel loops above use. */
#ifdef _OPENMP
#include <omp.h>
#endif
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * C = A * B for square block arrays under any law: (A*B)_ij is the sum over
 * k in B(i,j) of A_ik B_kj (the row-column rule with the law's support).
 * For law 0 this is oracle_square_star; the tests check law 2 against the
 * tensor product of two copies of the q = 2 rule.
 */
void oracle_square_law(int law, const unsigned char *edges, int q, int64_t bs, const double *A, const double *B, double *C)
{
    const int64_t n = q * bs;
    memset(C, 0, sizeof(double) * (size_t)(n * n));
    #define BLK(P, i, j, u, v) (P)[((i) * bs + (u)) * n + (j) * bs + (v)]
    for (int i = 0; i < q; ++i)
        for (int j = 0; j < q; ++j)
            for (int k = 0; k < q; ++k) {
                if (!oracle_in_support(law, edges, q, i, j, k)) continue;
                for (int64_t u = 0; u < bs; ++u)
                    for (int64_t v = 0; v < bs; ++v) {
                        double acc = 0.0;
                        for (int64_t w = 0; w < bs; ++w) acc += BLK(A, i, k, u, w) * BLK(B, k, j, w, v);
                        BLK(C, i, j, u, v) += acc;
                    }
            }
    #undef BLK
}

/* ---- algebraic attention (appendix "Attention Extension and Detailed Cost
 * Accounting") ------------------------------------------------------------
 *
 * One head of width d_h = q m is split into q groups of width m.  A query at
 * position p (type i = tau(p)) and a key at position u (type j = tau(u))
 * meet on the feature groups F(i,j) (eq. feature-set): {i} if i = j, else
 * {i, j} for the star law; every group for the dense law (ordinary
 * attention); for the tensor power, every beta whose bits each equal the
 * bit of i or of j (eq. tensor-square-feature-set).  The raw score is the
 * sum over a in F(i,j) of <Q_p^(a), K_u^(a)> (eq. attention-raw-score), the
 * score divides it by sqrt(|F(i,j)| m) (eqs. attention-support-size,
 * attention-score), keys after the query are masked (eq. causal-mask), and
 * the output is the softmax-weighted sum of the full value vectors
 * (eq. softmax-pv: dense value aggregation).
 *
 * Layouts: token-major rows, head h at columns [h d_h, (h+1) d_h), group a of
 * a head at [a m, (a+1) m) within it.  Head h reads key/value head
 * h / (n_heads / n_kv) (grouped-query attention).
 */
int oracle_attn_in_group(int law, int i, int j, int a)
{
    if (law == ORACLE_LAW_DENSE) return 1;
    if (law == ORACLE_LAW_TENSOR2) {
        for (int bit = 0; bit < 30; ++bit) {
            const int b = (a >> bit) & 1, x = (i >> bit) & 1, y = (j >> bit) & 1;
            if (b != x && b != y) return 0;
        }
        return 1;
    }
    return a == i || a == j;
}

/* score of query row qr (type i) and key row kr (type j) of one head pair */
static double attn_score(int law, int q, int64_t m, int i, int j, const double *qr, const double *kr)
{
    double r = 0.0;
    int nf = 0;
    for (int a = 0; a < q; ++a) {
        if (!oracle_attn_in_group(law, i, j, a)) continue;
        ++nf;
        for (int64_t c = 0; c < m; ++c) r += qr[a * m + c] * kr[a * m + c];
    }
    return r / sqrt((double)nf * (double)m);
}

/* Causal attention over B sequences of S positions (Alg. attention-training,
 * forward): Q [B S, n_heads d_h], K, V [B S, n_kv d_h], O [B S, n_heads d_h];
 * pos_type[p] is the type of position p.  lse, if not NULL, receives
 * [B, n_heads, S] the natural log of the softmax denominator of each query,
 * log sum_{u <= p} exp(s_pu) (eq. softmax-pv).  Returns 0, or -1 for an
 * out-of-range type or a head count that does not divide. */
int oracle_attn_fwd(int q, int law, int64_t m, int n_heads, int n_kv, int64_t B, int64_t S,
                    const int32_t *pos_type, const double *Q, const double *K, const double *V, double *O,
                    double *lse)
{
    if (n_kv <= 0 || n_heads % n_kv) return -1;
    for (int64_t p = 0; p < S; ++p)
        if (pos_type[p] < 0 || pos_type[p] >= q) return -1;
    const int64_t dh = q * m, ldq = n_heads * dh, ldk = n_kv * dh;
    const int group = n_heads / n_kv;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int h = 0; h < n_heads; ++h) {
            const int hk = h / group;
            double *s = (double *)malloc(sizeof(double) * (size_t)S);
            for (int64_t p = 0; p < S; ++p) {
                const double *qr = Q + (b * S + p) * ldq + h * dh;
                double mx = -INFINITY;
                for (int64_t u = 0; u <= p; ++u) {
                    s[u] = attn_score(law, q, m, pos_type[p], pos_type[u], qr, K + (b * S + u) * ldk + hk * dh);
                    if (s[u] > mx) mx = s[u];
                }
                double den = 0.0;
                for (int64_t u = 0; u <= p; ++u) {
                    s[u] = exp(s[u] - mx);
                    den += s[u];
                }
                if (lse) lse[(b * n_heads + h) * S + p] = mx + log(den);
                double *o = O + (b * S + p) * ldq + h * dh;
                for (int64_t c = 0; c < dh; ++c) o[c] = 0.0;
                for (int64_t u = 0; u <= p; ++u) {
                    const double w = s[u] / den;
                    const double *vr = V + (b * S + u) * ldk + hk * dh;
                    for (int64_t c = 0; c < dh; ++c) o[c] += w * vr[c];
                }
            }
            free(s);
        }
    return 0;
}

/* One decode step (Alg. attention-decoding): sequence b has cache_len[b]
 * cached positions 0..cache_len[b]-1 (the new token's key and value already
 * appended) and its query is at position cache_len[b] - 1.  Q [B, n_heads
 * d_h]; K_cache, V_cache [B, S_max, n_kv d_h]; O [B, n_heads d_h]. */
int oracle_attn_decode(int q, int law, int64_t m, int n_heads, int n_kv, int64_t B, int64_t S_max,
                       const int32_t *pos_type, const int32_t *cache_len, const double *Q,
                       const double *Kc, const double *Vc, double *O)
{
    if (n_kv <= 0 || n_heads % n_kv) return -1;
    const int64_t dh = q * m, ldq = n_heads * dh, ldk = n_kv * dh;
    const int group = n_heads / n_kv;
    for (int64_t b = 0; b < B; ++b) {
        if (cache_len[b] < 1 || cache_len[b] > S_max) return -1;
        for (int64_t u = 0; u < cache_len[b]; ++u)
            if (pos_type[u] < 0 || pos_type[u] >= q) return -1;
    }
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < B; ++b)
        for (int h = 0; h < n_heads; ++h) {
            const int hk = h / group;
            const int64_t L = cache_len[b], p = L - 1;
            double *s = (double *)malloc(sizeof(double) * (size_t)L);
            const double *qr = Q + b * ldq + h * dh;
            double mx = -INFINITY;
            for (int64_t u = 0; u < L; ++u) {
                s[u] = attn_score(law, q, m, pos_type[p], pos_type[u], qr, Kc + (b * S_max + u) * ldk + hk * dh);
                if (s[u] > mx) mx = s[u];
            }
            double den = 0.0;
            for (int64_t u = 0; u < L; ++u) {
                s[u] = exp(s[u] - mx);
                den += s[u];
            }
            double *o = O + b * ldq + h * dh;
            for (int64_t c = 0; c < dh; ++c) o[c] = 0.0;
            for (int64_t u = 0; u < L; ++u) {
                const double w = s[u] / den;
                const double *vr = Vc + (b * S_max + u) * ldk + hk * dh;
                for (int64_t c = 0; c < dh; ++c) o[c] += w * vr[c];
            }
            free(s);
        }
    return 0;
}
