"""Pins for the CPU oracle: checks against what the paper and mathematics fix.

Every test here runs on the CPU.  None of them re-types the oracle's own loop:
each compares it with a different formulation (the square display, a masked
dense product through numpy's BLAS, a brute-force enumeration of the basis
products, the semidirect formula, closed-form counts, invariants such as
associativity and the adjoint identity, finite differences, tabulated and
series values of the normal distribution function, scipy's ndtr,
torch's bfloat16 cast) or with hand-evaluated golden values.
"""

import math
import os

import numpy as np
import pytest

import oracle
from oracle import Alg

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            out[key] = np.array([float(v) for v in vals])
    return out


def rng(*seed):
    return np.random.default_rng(list(seed))


def square_typed(q, bs, A, B, law="star"):
    """A *_q B through the typed projection: row block i of A has type i."""
    alg = Alg.equal(q, q * bs, q * bs, law)
    t = np.repeat(np.arange(q), bs).astype(np.int32)
    Y, _, _, _ = oracle.proj_fwd(alg, t, A, B)
    return Y


def masked_dense_fwd(alg, t, X, W):
    """Independent formulation: Y[I_i] = X[I_i] (W . Mask_i),
    Mask_i[kk, n] = [group(kk) in {i, group(n)}] (Sec. 4, eqs. typed-diag/-off)."""
    gk = np.repeat(np.arange(alg.q), alg.s)
    gn = np.repeat(np.arange(alg.q), alg.r)
    Y = np.zeros((X.shape[0], alg.N))
    for i in range(alg.q):
        rows = np.nonzero(t == i)[0]
        if alg.law == "dense":
            mask = np.ones((alg.K, alg.N))
        else:
            mask = ((gk[:, None] == i) | (gk[:, None] == gn[None, :])).astype(float)
        Y[rows] = X[rows] @ (W * mask)
    return Y


# ---- P1: the q = 2 display ---------------------------------------------------

def test_q2_display_golden_scalars():
    g = _read_golden("q2_display_scalar.txt")
    X = g["X"].reshape(2, 2)
    W = g["W"].reshape(2, 2)
    t = np.array([0, 1], dtype=np.int32)
    Y, _, _, _ = oracle.proj_fwd(Alg(2, (1, 1), (1, 1), "star"), t, X, W)
    np.testing.assert_array_equal(Y.ravel(), g["STAR"])
    Yd, _, _, _ = oracle.proj_fwd(Alg(2, (1, 1), (1, 1), "dense"), t, X, W)
    np.testing.assert_array_equal(Yd.ravel(), g["DENSE"])


@pytest.mark.parametrize("bs", [1, 3, 8])
def test_q2_display_blocks(bs):
    """Sec. 1 eq. six-product with matrix blocks: type-1 rows give
    [A Wa, A Wu + U Wd], type-2 rows give [V Wa + D Wv, D Wd]."""
    g = rng(1, bs)
    A, U, V, D = (g.standard_normal((bs, bs)) for _ in range(4))
    Wa, Wu, Wv, Wd = (g.standard_normal((bs, bs)) for _ in range(4))
    X = np.block([[A, U], [V, D]])
    W = np.block([[Wa, Wu], [Wv, Wd]])
    expect = np.block([[A @ Wa, A @ Wu + U @ Wd], [V @ Wa + D @ Wv, D @ Wd]])
    got = square_typed(2, bs, X, W)
    np.testing.assert_allclose(got, expect, rtol=0, atol=1e-12)
    # the two removed products really are absent: perturbing U.Wv's factor
    # pair only through that product changes nothing
    W2 = np.block([[Wa, Wu], [Wv + 1.0, Wd]])
    got2 = square_typed(2, bs, X, W2)
    np.testing.assert_allclose(got2[:bs], got[:bs], rtol=0, atol=0)


def test_q2_interleaved_rows():
    """Rows of the two types interleaved (t = b mod 2) as in a sequence."""
    g = rng(2)
    M, s = 10, (3, 5)
    alg = Alg(2, s, (4, 2))
    X = g.standard_normal((M, alg.K))
    W = g.standard_normal((alg.K, alg.N))
    t = (np.arange(M) % 2).astype(np.int32)
    Y, _, _, _ = oracle.proj_fwd(alg, t, X, W)
    x1, x2 = X[:, :3], X[:, 3:]
    Wa, Wu, Wv, Wd = W[:3, :4], W[:3, 4:], W[3:, :4], W[3:, 4:]
    for b in range(M):
        if t[b] == 0:
            exp = np.concatenate([x1[b] @ Wa, x1[b] @ Wu + x2[b] @ Wd])
        else:
            exp = np.concatenate([x1[b] @ Wa + x2[b] @ Wv, x2[b] @ Wd])
        np.testing.assert_allclose(Y[b], exp, atol=1e-12)


# ---- P2, P3: reductions to ordinary products --------------------------------

@pytest.mark.parametrize("law", ["star", "dense"])
def test_q1_is_gemm(law):
    g = rng(3)
    X, W = g.standard_normal((7, 6)), g.standard_normal((6, 5))
    Y, _, _, _ = oracle.proj_fwd(Alg(1, (6,), (5,), law), np.zeros(7, np.int32), X, W)
    np.testing.assert_allclose(Y, X @ W, atol=1e-12)


@pytest.mark.parametrize("q,s,r", [(2, (4, 4), (3, 3)), (3, (2, 5, 1), (4, 1, 3)), (4, (2,) * 4, (3,) * 4)])
def test_dense_law_is_gemm(q, s, r):
    g = rng(4, q)
    alg = Alg(q, s, r, "dense")
    X, W = g.standard_normal((9, alg.K)), g.standard_normal((alg.K, alg.N))
    t = g.integers(0, q, 9).astype(np.int32)
    Y, _, _, ppt = oracle.proj_fwd(alg, t, X, W)
    np.testing.assert_allclose(Y, X @ W, atol=1e-12)
    assert list(ppt) == [q * q] * q


# ---- P4: masked dense --------------------------------------------------------

@pytest.mark.parametrize("q,s,r", [(2, (3, 5), (4, 2)), (3, (2, 5, 1), (4, 1, 3)),
                                   (5, (1, 2, 3, 2, 1), (2, 2, 1, 3, 4)), (4, (4,) * 4, (4,) * 4)])
def test_masked_dense_forward(q, s, r):
    g = rng(5, q)
    alg = Alg(q, s, r)
    M = 23
    X, W = g.standard_normal((M, alg.K)), g.standard_normal((alg.K, alg.N))
    t = g.integers(0, q, M).astype(np.int32)
    Y, _, _, _ = oracle.proj_fwd(alg, t, X, W)
    np.testing.assert_allclose(Y, masked_dense_fwd(alg, t, X, W), atol=1e-12)


def test_masked_dense_backward():
    """dX[I_i] = dY[I_i] (W . Mask_i)^T ; dW = sum_i (X[I_i]^T dY[I_i]) . Mask_i."""
    q, s, r = 3, (2, 4, 3), (3, 2, 5)
    alg = Alg(q, s, r)
    g = rng(6)
    M = 17
    X, W, dY = g.standard_normal((M, alg.K)), g.standard_normal((alg.K, alg.N)), g.standard_normal((M, alg.N))
    t = g.integers(0, q, M).astype(np.int32)
    gk = np.repeat(np.arange(q), s)
    gn = np.repeat(np.arange(q), r)
    dX_exp = np.zeros((M, alg.K))
    dW_exp = np.zeros((alg.K, alg.N))
    for i in range(q):
        rows = np.nonzero(t == i)[0]
        mask = ((gk[:, None] == i) | (gk[:, None] == gn[None, :])).astype(float)
        dX_exp[rows] = dY[rows] @ (W * mask).T
        dW_exp += (X[rows].T @ dY[rows]) * mask
    np.testing.assert_allclose(oracle.proj_bwd_data(alg, t, dY, W), dX_exp, atol=1e-12)
    dW, db = oracle.proj_bwd_weight(alg, t, X, dY)
    np.testing.assert_allclose(dW, dW_exp, atol=1e-12)
    np.testing.assert_allclose(db, dY.sum(0), atol=1e-12)


# ---- P5: brute-force structure constants of Q_q (x) M_b ----------------------

def _basis_product_table(q):
    """Nonzero basis products of Q_q (eq. graph-basis-products):
    e_i e_i = e_i, e_i a_ij = a_ij, a_ij e_j = a_ij.  Slots are (row, col)
    pairs: (i,i) is the vertex e_i, (i,j) the edge a_ij.  Returns a dict
    (slot_x, slot_w) -> slot of the product."""
    table = {}
    for i in range(q):
        table[((i, i), (i, i))] = (i, i)
        for j in range(q):
            if j != i:
                table[((i, i), (i, j))] = (i, j)
                table[((i, j), (j, j))] = (i, j)
    return table


@pytest.mark.parametrize("q,bs", [(1, 2), (2, 1), (2, 2), (3, 2), (4, 1), (4, 3)])
def test_bruteforce_structure_constants(q, bs):
    """Expand A and B over the basis slot (x) E_uv of Q_q (x) M_b and sum every
    nonzero basis product, then compare with the oracle's typed projection and
    its square-rule routine."""
    table = _basis_product_table(q)
    assert len(table) == 2 * q * q - q  # eq. q-rank
    g = rng(7, q, bs)
    n = q * bs
    A, B = g.standard_normal((n, n)), g.standard_normal((n, n))
    C = np.zeros((n, n))
    for (sx, sw), sc in table.items():
        for u in range(bs):
            for v in range(bs):
                a = A[sx[0] * bs + u, sx[1] * bs + v]
                for z in range(bs):  # E_uv E_vz = E_uz
                    C[sc[0] * bs + u, sc[1] * bs + z] += a * B[sw[0] * bs + v, sw[1] * bs + z]
    np.testing.assert_allclose(square_typed(q, bs, A, B), C, atol=1e-12)
    np.testing.assert_allclose(oracle.square_star(q, bs, A, B), C, atol=1e-12)
    assert sum(oracle.products_per_type("star", q, i) for i in range(q)) == len(table)


# ---- golden: the Q_3 square rule ------------------------------------------------

def test_q3_square_rule_golden():
    g = _read_golden("q3_square_rule.txt")
    A, B = g["A"].reshape(3, 3), g["B"].reshape(3, 3)
    np.testing.assert_array_equal(square_typed(3, 1, A, B).ravel(), g["STAR"])
    np.testing.assert_array_equal(oracle.square_star(3, 1, A, B).ravel(), g["STAR"])


# ---- P6, P8: associativity, unit, semidirect form ----------------------------

@pytest.mark.parametrize("q", [2, 3, 4, 5])
def test_associativity_and_unit(q):
    bs = 3
    g = rng(8, q)
    n = q * bs
    A, B, C = (g.standard_normal((n, n)) for _ in range(3))
    lhs = square_typed(q, bs, square_typed(q, bs, A, B), C)
    rhs = square_typed(q, bs, A, square_typed(q, bs, B, C))
    np.testing.assert_allclose(lhs, rhs, atol=1e-11)
    E = np.eye(n)
    np.testing.assert_allclose(square_typed(q, bs, E, B), B, atol=0)
    np.testing.assert_allclose(square_typed(q, bs, A, E), A, atol=0)
    # the ordinary product is associative too, but the two laws differ
    assert not np.allclose(square_typed(q, bs, A, B), A @ B)


def _semidirect(q, bs, A, B):
    """App. "Direct Associativity Check": (d,n)*(d',n') = (dd', dn' + nd')
    with (dn')_ij = d_i n'_ij and (nd')_ij = n_ij d'_j, over matrix blocks."""
    blk = lambda P, i, j: P[i * bs:(i + 1) * bs, j * bs:(j + 1) * bs]
    out = np.zeros_like(A)
    for i in range(q):
        blk(out, i, i)[:] = blk(A, i, i) @ blk(B, i, i)
    for i in range(q):
        for j in range(q):
            if i != j:
                blk(out, i, j)[:] = blk(A, i, i) @ blk(B, i, j) + blk(A, i, j) @ blk(B, j, j)
    return out


@pytest.mark.parametrize("q", [2, 3, 5])
def test_semidirect_form(q):
    bs = 2
    g = rng(9, q)
    A, B = g.standard_normal((q * bs, q * bs)), g.standard_normal((q * bs, q * bs))
    np.testing.assert_allclose(square_typed(q, bs, A, B), _semidirect(q, bs, A, B), atol=1e-12)


# ---- P7: composition of typed projections ------------------------------------

@pytest.mark.parametrize("q,law", [(2, "star"), (3, "star"), (4, "star"), (4, "tensor2")])
def test_composition(q, law):
    """eq. association-intro / general-associativity, rectangular groups:
    Phi_{W2}(Phi_{W1}(X)) = Phi_{W1 * W2}(X), where W1 * W2 is the algebra
    product of the two banks (row group i of W1 is a type-i row)."""
    g = rng(10, q)
    s = tuple(int(v) for v in g.integers(1, 4, q))
    r1 = tuple(int(v) for v in g.integers(1, 4, q))
    r2 = tuple(int(v) for v in g.integers(1, 4, q))
    a1, a2, a12 = Alg(q, s, r1, law), Alg(q, r1, r2, law), Alg(q, s, r2, law)
    M = 13
    X = g.standard_normal((M, a1.K))
    W1, W2 = g.standard_normal((a1.K, a1.N)), g.standard_normal((a2.K, a2.N))
    t = g.integers(0, q, M).astype(np.int32)
    t_w1 = np.repeat(np.arange(q), s).astype(np.int32)
    W12, _, _, _ = oracle.proj_fwd(a2, t_w1, W1, W2)  # rows of W1 in group i have type i
    Y1, _, _, _ = oracle.proj_fwd(a1, t, X, W1)
    lhs, _, _, _ = oracle.proj_fwd(a2, t, Y1, W2)
    rhs, _, _, _ = oracle.proj_fwd(a12, t, X, W12)
    np.testing.assert_allclose(lhs, rhs, atol=1e-11)


# ---- P9, P10: identity bank, row locality ------------------------------------

@pytest.mark.parametrize("q", [1, 2, 3, 4])
def test_identity_bank(q):
    g = rng(11, q)
    s = tuple(int(v) for v in g.integers(1, 5, q))
    alg = Alg(q, s, s)
    X = g.standard_normal((11, alg.K))
    t = g.integers(0, q, 11).astype(np.int32)
    Y, _, _, _ = oracle.proj_fwd(alg, t, X, np.eye(alg.K))
    np.testing.assert_array_equal(Y, X)


def test_row_locality():
    """Prop. "Causality": the projection acts on each row independently."""
    alg = Alg(3, (2, 3, 4), (3, 3, 2))
    g = rng(12)
    M = 9
    X, W = g.standard_normal((M, alg.K)), g.standard_normal((alg.K, alg.N))
    t = (np.arange(M) % 3).astype(np.int32)
    bias = g.standard_normal(alg.N)
    Y0, _, _, _ = oracle.proj_fwd(alg, t, X, W, bias, "gelu")
    for b in range(M):
        X2 = X.copy()
        X2[b] += g.standard_normal(alg.K)
        Y2, _, _, _ = oracle.proj_fwd(alg, t, X2, W, bias, "gelu")
        changed = np.nonzero(np.any(Y2 != Y0, axis=1))[0]
        assert list(changed) == [b]
        # and the result of a row does not depend on its neighbours' presence
        Yb, _, _, _ = oracle.proj_fwd(alg, t[b:b + 1], X[b:b + 1], W, bias, "gelu")
        np.testing.assert_array_equal(Yb[0], Y0[b])


# ---- P11: backward -------------------------------------------------------------

@pytest.mark.parametrize("law", ["star", "dense", "tensor2"])
def test_adjoint_identity(law):
    """<Phi(X,W), G> = <X, dX> = <W, dW>, exact by bilinearity (App. VJPs)."""
    alg = Alg(4, (2, 3, 1, 2), (3, 1, 2, 2), law)
    g = rng(13)
    M = 15
    X, W, G = g.standard_normal((M, alg.K)), g.standard_normal((alg.K, alg.N)), g.standard_normal((M, alg.N))
    t = g.integers(0, 4, M).astype(np.int32)
    Y, _, _, _ = oracle.proj_fwd(alg, t, X, W)
    dX = oracle.proj_bwd_data(alg, t, G, W)
    dW, _ = oracle.proj_bwd_weight(alg, t, X, G)
    a, b, c = np.sum(Y * G), np.sum(X * dX), np.sum(W * dW)
    assert abs(a - b) < 1e-10 * max(1, abs(a)) and abs(a - c) < 1e-10 * max(1, abs(a))
    # the adjoint pairs fail for a wrong gradient: the dense gradient under the star law
    if law == "star":
        dXd = oracle.proj_bwd_data(Alg(alg.q, alg.s, alg.r, "dense"), t, G, W)
        assert abs(np.sum(X * dXd) - a) > 1e-3


def test_finite_differences_through_activation():
    """Central differences of L = <G, Phi_W2(act(Phi_W1(X) + b1)) + b2> against
    the chained VJPs (act' applied to the pre-activation)."""
    up, down = Alg(2, (2, 3), (3, 2)), Alg(2, (3, 2), (2, 2))
    g = rng(14)
    M = 5
    X = g.standard_normal((M, up.K))
    W1, W2 = g.standard_normal((up.K, up.N)) * 0.7, g.standard_normal((down.K, down.N)) * 0.7
    b1, b2 = g.standard_normal(up.N), g.standard_normal(down.N)
    G = g.standard_normal((M, down.N))
    t = (np.arange(M) % 2).astype(np.int32)

    def loss(X_, W1_, W2_, b1_, b2_):
        _, _, Y = oracle.ffn_fwd(up, down, t, X_, W1_, b1_, W2_, b2_, "gelu", mirror_bf16=False)
        return float(np.sum(G * Y))

    Z, H, _ = oracle.ffn_fwd(up, down, t, X, W1, b1, W2, b2, "gelu", mirror_bf16=False)
    gr = oracle.ffn_bwd(up, down, t, X, Z, H, W1, W2, G, "gelu", mirror_bf16=False)
    h = 1e-5
    for name, arr, grad in [("X", X, gr["dX"]), ("W1", W1, gr["dW_up"]), ("W2", W2, gr["dW_down"]),
                            ("b1", b1, gr["db_up"]), ("b2", b2, gr["db_down"])]:
        flat = arr.reshape(-1)
        for idx in range(flat.size):
            old = flat[idx]
            flat[idx] = old + h
            lp = loss(X, W1, W2, b1, b2)
            flat[idx] = old - h
            lm = loss(X, W1, W2, b1, b2)
            flat[idx] = old
            fd = (lp - lm) / (2 * h)
            assert abs(fd - grad.reshape(-1)[idx]) < 1e-6 * max(1.0, abs(fd)), (name, idx)


def test_bwd_weight_entries_match_full():
    alg = Alg(3, (4, 2, 3), (2, 5, 3))
    g = rng(15)
    M = 19
    X, dY = g.standard_normal((M, alg.K)), g.standard_normal((M, alg.N))
    t = g.integers(0, 3, M).astype(np.int32)
    t[t == 1] = 0  # an absent type: its off-diagonal row of blocks is zero
    dW, _ = oracle.proj_bwd_weight(alg, t, X, dY)
    kk, nn = np.meshgrid(np.arange(alg.K), np.arange(alg.N), indexing="ij")
    ent = oracle.bwd_weight_entries(alg, t, X, dY, kk.ravel(), nn.ravel())
    np.testing.assert_allclose(ent.reshape(alg.K, alg.N), dW, atol=1e-12)
    # type 1 absent: W_1j (j != 1) gets no gradient
    np.testing.assert_array_equal(dW[4:6, :2], 0)
    np.testing.assert_array_equal(dW[4:6, 7:], 0)
    assert np.all(dW[4:6, 2:7] != 0)


# ---- P12: counts ---------------------------------------------------------------

@pytest.mark.parametrize("q", [1, 2, 3, 4, 8, 16])
def test_product_counts(q):
    for i in range(q):
        assert oracle.products_per_type("star", q, i) == 2 * q - 1
        assert oracle.products_per_type("dense", q, i) == q * q
    # rho_q = (2q-1)/q^2 for equal groups (eq. rho)
    alg = Alg.equal(q, 8 * q, 4 * q)
    for i in range(q):
        assert oracle.row_macs(alg, i) * q * q == (2 * q - 1) * alg.K * alg.N


def test_unequal_row_cost_and_batch_cost():
    """eq. unequal-row-cost C_i = D_diag + s_i (N - r_i) and
    eq. rectangular-batch-cost, against the MACs the oracle visits."""
    s, r = (2, 5, 3, 1), (4, 1, 2, 6)
    alg = Alg(4, s, r)
    D_diag = sum(a * b for a, b in zip(s, r))
    N = sum(r)
    for i in range(4):
        assert oracle.row_macs(alg, i) == D_diag + s[i] * (N - r[i])
    g = rng(16)
    M = 31
    t = g.integers(0, 4, M).astype(np.int32)
    X, W = g.standard_normal((M, alg.K)), g.standard_normal((alg.K, alg.N))
    _, _, macs, _ = oracle.proj_fwd(alg, t, X, W)
    Mi = np.bincount(t, minlength=4)
    assert macs == M * D_diag + sum(int(Mi[i]) * s[i] * (N - r[i]) for i in range(4))


# ---- P13: activations ------------------------------------------------------------

def _phi_table():
    """Tabulated values of the standard normal distribution function."""
    out = []
    with open(os.path.join(GOLDEN, "normal_cdf.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                x, p = line.split()
                out.append((float(x), float(p)))
    return out


def _dec_phi(x, prec=60):
    """Phi(x) = (1 + erf(x / sqrt 2)) / 2 in decimal arithmetic, erf by its
    Maclaurin series 2/sqrt(pi) sum_n (-1)^n x^(2n+1) / (n! (2n+1)) (no libm;
    pi by the Gauss-Legendre iteration)."""
    from decimal import Decimal, getcontext
    getcontext().prec = prec
    a, b, t, p = Decimal(1), Decimal(1) / Decimal(2).sqrt(), Decimal(1) / 4, Decimal(1)
    for _ in range(8):
        an = (a + b) / 2
        b = (a * b).sqrt()
        t -= p * (a - an) ** 2
        a, p = an, 2 * p
    pi = (a + b) ** 2 / (4 * t)
    u = Decimal(repr(float(x))) / Decimal(2).sqrt()
    term, total, n = u, u, 0
    while True:
        n += 1
        term = -term * u * u / n
        add = term / (2 * n + 1)
        total += add
        if abs(add) < Decimal(10) ** (-prec + 5):
            break
    erf = 2 / pi.sqrt() * total
    return (1 + erf) / 2, pi


def test_gelu_erf_form_against_tabulated_phi():
    """GELU(z) = z Phi(z) and GELU'(z) = Phi(z) + z phi(z) at tabulated points
    of Phi (both signs: Phi(-x) = 1 - Phi(x)); phi(z) = exp(-z^2/2)/sqrt(2 pi)."""
    for x, P in _phi_table():
        for z, Pz in ((x, P), (-x, 1.0 - P)):
            assert abs(oracle.act("gelu", z)[()] - z * Pz) <= 2e-15 * max(1.0, abs(z))
            dens = math.exp(-0.5 * z * z) / math.sqrt(2 * math.pi)
            assert abs(oracle.act_grad("gelu", z)[()] - (Pz + z * dens)) <= 2e-15 * max(1.0, abs(z))
    assert oracle.act("gelu", 0.0)[()] == 0.0
    assert oracle.act_grad("gelu", 0.0)[()] == 0.5


def test_gelu_erf_form_against_ndtr():
    """The same functions against scipy's normal distribution function (the
    Cephes ndtr, not libm's erf) on a dense grid and the tails.  Absolute
    bound: in the far negative tail 1 + erf(z / sqrt 2) cancels to a few ulps
    of 1, so the oracle is accurate to ~1e-16 absolute there, not relative."""
    from scipy.special import ndtr
    zs = np.concatenate([np.linspace(-12, 12, 4801), [-40.0, -20.0, 20.0, 40.0, 1e-8, -1e-8]])
    np.testing.assert_allclose(oracle.act("gelu", zs), zs * ndtr(zs), rtol=1e-13, atol=1e-14)
    dens = np.exp(-0.5 * zs * zs) / np.sqrt(2 * np.pi)
    np.testing.assert_allclose(oracle.act_grad("gelu", zs), ndtr(zs) + zs * dens, rtol=1e-12, atol=1e-15)


def test_gelu_erf_form_against_decimal_series():
    """And against Phi evaluated in 60-digit decimal arithmetic from erf's
    power series, on points of [-6, 6]."""
    for z in np.linspace(-6, 6, 49):
        phi, _ = _dec_phi(z)
        assert abs(oracle.act("gelu", z)[()] - z * float(phi)) <= 1e-15 * max(1.0, abs(z))


def _dec_gelu_tanh(z, prec=50):
    """Tanh-form GELU 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))) and its
    derivative in decimal arithmetic: tanh(u) = (e^(2u) - 1) / (e^(2u) + 1) with
    the decimal module's exp, and d/dz = 0.5 (1 + t) + 0.5 z (1 - t^2) u'(z),
    u'(z) = sqrt(2/pi) (1 + 3 * 0.044715 z^2)."""
    from decimal import Decimal, getcontext
    _, pi = _dec_phi(0.0, prec)
    getcontext().prec = prec
    zd = Decimal(repr(float(z)))
    c = (2 / pi).sqrt()
    k = Decimal("0.044715")
    u = c * (zd + k * zd ** 3)
    e = (2 * u).exp()
    t = (e - 1) / (e + 1)
    val = zd * (1 + t) / 2
    du = c * (1 + 3 * k * zd * zd)
    der = (1 + t) / 2 + zd * (1 - t * t) * du / 2
    return float(val), float(der)


def test_gelu_tanh_form_against_decimal():
    for z in np.concatenate([np.linspace(-8, 8, 65), [0.5, -0.5, 1.0, 2.0]]):
        val, der = _dec_gelu_tanh(z)
        assert abs(oracle.act("gelu_tanh", z)[()] - val) <= 2e-15 * max(1.0, abs(val))
        assert abs(oracle.act_grad("gelu_tanh", z)[()] - der) <= 1e-14
    # worked value: z = 1, u = sqrt(2/pi) * 1.044715 = 0.83356..., tanh(u) =
    # 0.68238..., GELU_tanh(1) = 0.5 (1 + tanh u) = 0.84119...
    assert abs(oracle.act("gelu_tanh", 1.0)[()] - 0.8411919906082768) < 1e-15


def test_gelu_tanh_form_gap_to_erf_form():
    """The tanh form differs from the exact form by at most 4.8e-4 (the
    largest gap, 4.73e-4, sits near |z| = 2.70), and is not the same function."""
    zs = np.linspace(-12, 12, 24001)
    gap = np.abs(oracle.act("gelu_tanh", zs) - oracle.act("gelu", zs))
    assert gap.max() <= 4.8e-4
    assert gap.max() >= 4.6e-4
    assert abs(abs(zs[gap.argmax()]) - 2.70) < 0.02


def test_silu_against_scipy():
    """SiLU z sigma(z), with scipy's logistic function as the reference."""
    from scipy.special import expit
    zs = np.linspace(-30, 30, 241)
    np.testing.assert_allclose(oracle.act("silu", zs), zs * expit(zs), rtol=1e-14, atol=1e-300)


@pytest.mark.parametrize("kind", ["gelu", "gelu_tanh", "silu", "none"])
def test_activation_gradient_fd(kind):
    h = 1e-6
    for z in np.linspace(-6, 6, 61):
        fd = (oracle.act(kind, z + h)[()] - oracle.act(kind, z - h)[()]) / (2 * h)
        assert abs(fd - oracle.act_grad(kind, z)[()]) < 1e-8


def test_bias_and_activation_applied():
    """Z = X W + bias through an identity bank, then Y = Z Phi(Z) with Phi
    from scipy's ndtr."""
    from scipy.special import ndtr
    alg = Alg(2, (3, 3), (3, 3))
    g = rng(17)
    X = g.standard_normal((6, 6))
    bias = g.standard_normal(6)
    t = (np.arange(6) % 2).astype(np.int32)
    Y, Z, _, _ = oracle.proj_fwd(alg, t, X, np.eye(6), bias, "gelu", want_z=True)
    np.testing.assert_allclose(Z, X + bias, atol=1e-15)
    np.testing.assert_allclose(Y, Z * ndtr(Z), atol=1e-15)


# ---- P14: bfloat16 rounding -----------------------------------------------------------

def test_round_bf16_against_torch():
    torch = pytest.importorskip("torch")
    import synth
    g = rng(18)
    x = np.concatenate([
        g.standard_normal(20000).astype(np.float32),
        (g.standard_normal(2000) * 1e-30).astype(np.float32),
        (g.standard_normal(2000) * 1e30).astype(np.float32),
        # exact ties: 8 significant bits plus a trailing half
        np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 2 ** -130 * 3, 0.0, -0.0], np.float32),
    ])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.round_bf16(x.astype(np.float64)), ref)
    np.testing.assert_array_equal(synth.bf16_bits_to_f64(synth.f32_to_bf16_bits(x)), ref)


# ---- P15: decode stack of one layer ------------------------------------------------------

def test_decode_one_layer_is_ffn_plus_residual():
    up, down = Alg(2, (4, 4), (8, 8)), Alg(2, (8, 8), (4, 4))
    g = rng(19)
    M = 3
    X = oracle.round_bf16(g.standard_normal((M, 8)))
    Wu, Wd = g.standard_normal((8, 16)) * 0.1, g.standard_normal((16, 8)) * 0.1
    bu, bd = g.standard_normal(16) * 0.1, g.standard_normal(8) * 0.1
    t = np.array([1, 0, 1], np.int32)
    h = oracle.decode_stack(up, down, t, X, [Wu], [bu], [Wd], [bd])
    _, _, f = oracle.ffn_fwd(up, down, t, X, Wu, bu, Wd, bd)
    np.testing.assert_allclose(h, X + f, atol=0)
    # the stack applies its layers in order
    h2 = oracle.decode_stack(up, down, t, X, [Wu, Wu * 0.5], [bu, bu], [Wd, Wd], [bd, bd])
    a = oracle.round_bf16(h)
    _, _, f2 = oracle.ffn_fwd(up, down, t, a, Wu * 0.5, bu, Wd, bd)
    np.testing.assert_allclose(h2, h + f2, atol=0)


def test_out_of_range_type_rejected():
    alg = Alg(2, (2, 2), (2, 2))
    with pytest.raises(ValueError):
        oracle.proj_fwd(alg, np.array([0, 2], np.int32), np.zeros((2, 4)), np.zeros((4, 4)))


# ---- the tensor-power law Q_2^(x)L (appendix "The Tensor-Square Candidate") ------

def _tensor_square_table():
    """Nonzero basis products of Q_2 (x) Q_2 built from two copies of the Q_2
    table: (x1 (x) x2)(w1 (x) w2) = (x1 w1) (x) (x2 w2).  A slot of the tensor
    square is a pair of group indices made of one bit per factor
    (g = g1 + 2 g2)."""
    t2 = _basis_product_table(2)
    comb = lambda a, b: (a[0] + 2 * b[0], a[1] + 2 * b[1])
    table = {}
    for (x1, w1), c1 in t2.items():
        for (x2, w2), c2 in t2.items():
            table[(comb(x1, x2), comb(w1, w2))] = comb(c1, c2)
    return table


@pytest.mark.parametrize("bs", [1, 2, 3])
def test_tensor_square_structure_constants(bs):
    """The tensor square of the two-group law, multiplied out from its Kronecker
    structure constants, is the oracle's law "tensor2" at q = 4, both as a
    square-rule product and through the typed projection; it has the 36
    block products the paper counts (4 x 1 + 8 x 2 + 4 x 4)."""
    table = _tensor_square_table()
    assert len(table) == 36
    q = 4
    g = rng(31, bs)
    n = q * bs
    A, B = g.standard_normal((n, n)), g.standard_normal((n, n))
    C = np.zeros((n, n))
    for (sx, sw), sc in table.items():
        for u in range(bs):
            for v in range(bs):
                a = A[sx[0] * bs + u, sx[1] * bs + v]
                for z in range(bs):
                    C[sc[0] * bs + u, sc[1] * bs + z] += a * B[sw[0] * bs + v, sw[1] * bs + z]
    np.testing.assert_allclose(oracle.square_law("tensor2", q, bs, A, B), C, atol=1e-12)
    np.testing.assert_allclose(square_typed(q, bs, A, B, law="tensor2"), C, atol=1e-12)
    assert sum(oracle.products_per_type("tensor2", q, i) for i in range(q)) == 36
    # a different law from the direct four-group one (28 products)
    assert sum(oracle.products_per_type("star", q, i) for i in range(q)) == 28
    assert not np.allclose(square_typed(q, bs, A, B, law="star"), C)


def test_tensor_power_one_is_the_two_group_law():
    g = rng(32)
    A, B = g.standard_normal((6, 6)), g.standard_normal((6, 6))
    np.testing.assert_allclose(square_typed(2, 3, A, B, law="tensor2"), square_typed(2, 3, A, B), atol=0)


@pytest.mark.parametrize("q", [4, 8])
def test_tensor_power_associativity_and_unit(q):
    """The tensor product of associative unital algebras is associative with
    the product of the units."""
    bs = 2
    g = rng(33, q)
    n = q * bs
    A, B, C = (g.standard_normal((n, n)) for _ in range(3))
    sq = lambda X, Y: square_typed(q, bs, X, Y, law="tensor2")
    np.testing.assert_allclose(sq(sq(A, B), C), sq(A, sq(B, C)), atol=1e-11)
    E = np.eye(n)
    np.testing.assert_allclose(sq(E, B), B, atol=0)
    np.testing.assert_allclose(sq(A, E), A, atol=0)


@pytest.mark.parametrize("L", [1, 2, 3])
def test_tensor_power_counts(L):
    """6^L block products in all (the recursive algorithm's count), and for
    equal widths with every type present the MACs of a type average (3/4)^L of
    the dense projection (eq. recursive-uniform-cost)."""
    q = 2 ** L
    assert sum(oracle.products_per_type("tensor2", q, i) for i in range(q)) == 6 ** L
    alg = Alg.equal(q, 4 * q, 8 * q, "tensor2")
    total = sum(oracle.row_macs(alg, i) for i in range(q))
    assert total * 4 ** L == 3 ** L * q * alg.K * alg.N


# ---- gated FFN (SwiGLU) compositions ---------------------------------------------

def test_swiglu_ffn_is_its_formula_and_gradients_match_fd():
    """The gated FFN through the typed projections equals the same FFN built
    from masked dense products; its backward matches central differences of a
    scalar loss (fp64, no bf16 mirroring)."""
    from scipy.special import expit
    up, down = Alg(2, (3, 5), (4, 6)), Alg(2, (4, 6), (3, 5))
    g = rng(41)
    M = 9
    X = g.standard_normal((M, up.K))
    Wg, Wu = g.standard_normal((up.K, up.N)), g.standard_normal((up.K, up.N))
    Wd = g.standard_normal((down.K, down.N))
    bg, bu, bd = g.standard_normal(up.N), g.standard_normal(up.N), g.standard_normal(down.N)
    t = g.integers(0, 2, M).astype(np.int32)
    Zg, Zu, H, Y = oracle.swiglu_ffn_fwd(up, down, t, X, Wg, bg, Wu, bu, Wd, bd, mirror_bf16=False)
    zg = masked_dense_fwd(up, t, X, Wg) + bg
    zu = masked_dense_fwd(up, t, X, Wu) + bu
    h = zg * expit(zg) * zu
    np.testing.assert_allclose(H, h, atol=1e-12)
    np.testing.assert_allclose(Y, masked_dense_fwd(down, t, h, Wd) + bd, atol=1e-11)
    G = g.standard_normal(Y.shape)
    grads = oracle.swiglu_ffn_bwd(up, down, t, X, Zg, Zu, H, Wg, Wu, Wd, G, mirror_bf16=False)
    loss = lambda **kw: np.sum(oracle.swiglu_ffn_fwd(up, down, t, kw.get("X", X), kw.get("Wg", Wg), bg,
                                                     kw.get("Wu", Wu), bu, kw.get("Wd", Wd), bd,
                                                     mirror_bf16=False)[3] * G)
    eps = 1e-6
    for name, arr, key in (("X", X, "dX"), ("Wg", Wg, "dW_gate"), ("Wu", Wu, "dW_up"), ("Wd", Wd, "dW_down")):
        for (a_, b_) in [(0, 0), (2, 3), (arr.shape[0] - 1, arr.shape[1] - 1)]:
            P_, Mn = arr.copy(), arr.copy()
            P_[a_, b_] += eps
            Mn[a_, b_] -= eps
            fd = (loss(**{name: P_}) - loss(**{name: Mn})) / (2 * eps)
            assert abs(fd - grads[key][a_, b_]) < 1e-6 * max(1, abs(fd)), (name, a_, b_)


def test_gated_decode_stack_is_layers_of_the_gated_ffn():
    """Without bf16 mirroring, one layer of the gated decode stack is the
    residual plus the gated FFN's output, and L layers compose."""
    up, down = Alg(2, (4, 4), (6, 6)), Alg(2, (6, 6), (4, 4))
    g = rng(43)
    M, L = 3, 2
    X = g.standard_normal((M, 8))
    t = np.array([0, 1, 1], np.int32)
    Ws = [[g.standard_normal((8, 12)) for _ in range(L)], [g.standard_normal((8, 12)) for _ in range(L)],
          [g.standard_normal((12, 8)) for _ in range(L)]]
    bs = [[g.standard_normal(12) for _ in range(L)], [g.standard_normal(12) for _ in range(L)],
          [g.standard_normal(8) for _ in range(L)]]
    h = X.copy()
    for l in range(L):
        _, _, _, Y = oracle.swiglu_ffn_fwd(up, down, t, h, Ws[0][l], bs[0][l], Ws[1][l], bs[1][l],
                                           Ws[2][l], bs[2][l], mirror_bf16=False)
        h = h + Y
    got = oracle.decode_stack_gated(up, down, t, X, Ws[0], bs[0], Ws[1], bs[1], Ws[2], bs[2],
                                    mirror_bf16=False)
    np.testing.assert_allclose(got, h, atol=1e-12)


# ---- P16: the graph algebra Q_G (Sec. "Graph Products with Exact Cost") -------------

def _random_graph(q, p, seed):
    """A directed graph on q vertices without self-loops, each edge present
    with probability p."""
    g = rng(40, q, seed)
    E = (g.random((q, q)) < p).astype(np.uint8)
    np.fill_diagonal(E, 0)
    return E


GRAPHS = [
    ("path3", np.array([[0, 1, 0], [0, 0, 1], [0, 0, 0]], np.uint8)),
    ("cycle4", np.array([[0, 1, 0, 0], [0, 0, 1, 0], [0, 0, 0, 1], [1, 0, 0, 0]], np.uint8)),
    ("star_out4", np.array([[0, 1, 1, 1], [0, 0, 0, 0], [0, 0, 0, 0], [0, 0, 0, 0]], np.uint8)),
    ("random5", _random_graph(5, 0.45, 1)),
    ("random6", _random_graph(6, 0.3, 2)),
]


def _graph_table(E):
    """Nonzero basis products of Q_G from eq. graph-basis-products: vertex
    slots (i,i) = e_i and edge slots (i,j) = a_ij for the edges i -> j of G,
    e_i e_i = e_i, e_i a_ij = a_ij, a_ij e_j = a_ij; every other product of
    basis elements (edge times edge, mismatched indices) vanishes."""
    q = E.shape[0]
    slots = [(i, i) for i in range(q)] + [(i, j) for i in range(q) for j in range(q) if E[i, j] and i != j]
    table = {}
    for x in slots:
        for w in slots:
            if x[0] == x[1] and w[0] == w[1] and x[0] == w[0]:
                table[(x, w)] = x                      # e_i e_i = e_i
            elif x[0] == x[1] and w[0] != w[1] and w[0] == x[0]:
                table[(x, w)] = w                      # e_i a_ij = a_ij
            elif x[0] != x[1] and w[0] == w[1] and x[1] == w[0]:
                table[(x, w)] = x                      # a_ij e_j = a_ij
    return slots, table


def _slot_mask(E, bs):
    q = E.shape[0]
    m = np.zeros((q * bs, q * bs))
    for i in range(q):
        for j in range(q):
            if i == j or E[i, j]:
                m[i * bs:(i + 1) * bs, j * bs:(j + 1) * bs] = 1
    return m


def _graph_alg(E, s, r):
    return Alg(E.shape[0], tuple(s), tuple(r), "graph", tuple(tuple(int(v) for v in row) for row in E))


@pytest.mark.parametrize("name,E", GRAPHS)
def test_graph_bruteforce_structure_constants(name, E):
    """Square product of Q_G (x) M_b from the basis products, against the
    oracle's square rule and its typed projection (row block i of A is a
    type-i token; non-slot blocks of A and W are zero)."""
    q, bs = E.shape[0], 2
    slots, table = _graph_table(E)
    g = rng(41, q)
    n = q * bs
    mask = _slot_mask(E, bs)
    A, B = g.standard_normal((n, n)) * mask, g.standard_normal((n, n)) * mask
    C = np.zeros((n, n))
    for (sx, sw), sc in table.items():
        for u in range(bs):
            for v in range(bs):
                a = A[sx[0] * bs + u, sx[1] * bs + v]
                for z in range(bs):
                    C[sc[0] * bs + u, sc[1] * bs + z] += a * B[sw[0] * bs + v, sw[1] * bs + z]
    np.testing.assert_allclose(oracle.square_law("graph", q, bs, A, B, edges=E), C, atol=1e-12)
    alg = Alg(q, (bs,) * q, (bs,) * q, "graph", tuple(map(tuple, E)))
    t = np.repeat(np.arange(q), bs).astype(np.int32)
    Y, _, _, ppt = oracle.proj_fwd(alg, t, A, B)
    np.testing.assert_allclose(Y, C, atol=1e-12)
    # the number of basis products is the exact bilinear rank |V| + 2|E| (eq. graph-rank)
    nE = int(E.sum())
    assert len(table) == q + 2 * nE
    assert sum(oracle.products_per_type("graph", q, i, edges=E) for i in range(q)) == q + 2 * nE
    for i in range(q):
        assert oracle.products_per_type("graph", q, i, edges=E) == 1 + 2 * int(E[i].sum())
        assert ppt[i] == 1 + 2 * int(E[i].sum())


@pytest.mark.parametrize("name,E", GRAPHS)
def test_graph_typed_rule_is_masked_dense(name, E):
    """Independent formulation of the typed rule (eqs. graph-product-vertex,
    graph-product-edge): Y[I_i] = X[I_i] (W . Mask_i) with Mask_i[kk, n] = 1
    when group(n) = i and group(kk) = i, or group(n) = j for an edge i -> j
    and group(kk) in {i, j}; the gradients are the same masked products."""
    q = E.shape[0]
    s, r = [2 + (g % 3) for g in range(q)], [3 - (g % 2) for g in range(q)]
    alg = _graph_alg(E, s, r)
    gk = np.repeat(np.arange(q), s)
    gn = np.repeat(np.arange(q), r)
    g = rng(42, q)
    M = 23
    X, W, G = g.standard_normal((M, alg.K)), g.standard_normal((alg.K, alg.N)), g.standard_normal((M, alg.N))
    t = g.integers(0, q, M).astype(np.int32)
    Y, _, _, _ = oracle.proj_fwd(alg, t, X, W)
    dX = oracle.proj_bwd_data(alg, t, G, W)
    dW, db = oracle.proj_bwd_weight(alg, t, X, G)
    Yr, dXr, dWr = np.zeros_like(Y), np.zeros_like(dX), np.zeros_like(dW)
    for i in range(q):
        out_ok = (gn == i) | E[i][gn].astype(bool)
        mask = (out_ok[None, :] & ((gk[:, None] == i) | (gk[:, None] == gn[None, :]))).astype(float)
        rows = np.nonzero(t == i)[0]
        Yr[rows] = X[rows] @ (W * mask)
        dXr[rows] = G[rows] @ (W * mask).T
        dWr += (X[rows].T @ G[rows]) * mask
    np.testing.assert_allclose(Y, Yr, atol=1e-12)
    np.testing.assert_allclose(dX, dXr, atol=1e-12)
    np.testing.assert_allclose(dW, dWr, atol=1e-12)
    np.testing.assert_allclose(db, G.sum(0), atol=1e-12)


def test_graph_special_cases():
    """The complete graph is the star law Q_q; the empty graph keeps only the
    vertex products (a type-i row's output is x_i W_ii in group i, zero in the
    groups that are not its slots)."""
    q = 4
    alg_s = Alg(q, (3, 2, 2, 1), (2, 3, 1, 2), "star")
    full = np.ones((q, q), np.uint8) - np.eye(q, dtype=np.uint8)
    g = rng(43)
    M = 17
    X, W = g.standard_normal((M, alg_s.K)), g.standard_normal((alg_s.K, alg_s.N))
    t = g.integers(0, q, M).astype(np.int32)
    Ys, _, _, _ = oracle.proj_fwd(alg_s, t, X, W)
    Yg, _, _, _ = oracle.proj_fwd(_graph_alg(full, alg_s.s, alg_s.r), t, X, W)
    np.testing.assert_array_equal(Yg, Ys)
    Ye, _, _, _ = oracle.proj_fwd(_graph_alg(np.zeros((q, q), np.uint8), alg_s.s, alg_s.r), t, X, W)
    S = np.concatenate([[0], np.cumsum(alg_s.s)])
    R = np.concatenate([[0], np.cumsum(alg_s.r)])
    ref = np.zeros_like(Ye)
    for b in range(M):
        i = t[b]
        ref[b, R[i]:R[i + 1]] = X[b, S[i]:S[i + 1]] @ W[S[i]:S[i + 1], R[i]:R[i + 1]]
    np.testing.assert_allclose(Ye, ref, atol=1e-12)


@pytest.mark.parametrize("name,E", GRAPHS)
def test_graph_associativity_unit_composition(name, E):
    """Q_G is associative and unital (Proposition "Structure"): on slot-
    supported block arrays (A * B) * C = A * (B * C) and the sum of the
    vertex identities is the unit; and the typed projection composes,
    Phi_W2(Phi_W1(X)) = Phi_{W1 * W2}(X), when the inputs' non-slot groups
    are zero."""
    q, bs = E.shape[0], 3
    n = q * bs
    mask = _slot_mask(E, bs)
    g = rng(44, q)
    A, B, C = (g.standard_normal((n, n)) * mask for _ in range(3))
    sq = lambda P, Q: oracle.square_law("graph", q, bs, P, Q, edges=E)
    np.testing.assert_allclose(sq(sq(A, B), C), sq(A, sq(B, C)), atol=1e-11)
    I = np.eye(n)
    np.testing.assert_allclose(sq(I, B), B, atol=0)
    np.testing.assert_allclose(sq(A, I), A, atol=0)
    alg = Alg(q, (bs,) * q, (bs,) * q, "graph", tuple(map(tuple, E)))
    M = 19
    t = g.integers(0, q, M).astype(np.int32)
    X = g.standard_normal((M, n))
    for b in range(M):  # a type-i token carries only its slots
        X[b] *= mask[t[b] * bs]
    W1, W2 = g.standard_normal((n, n)) * mask, g.standard_normal((n, n)) * mask
    Y1, _, _, _ = oracle.proj_fwd(alg, t, X, W1)
    Y2, _, _, _ = oracle.proj_fwd(alg, t, Y1, W2)
    Y12, _, _, _ = oracle.proj_fwd(alg, t, X, sq(W1, W2))
    np.testing.assert_allclose(Y2, Y12, atol=1e-11)


def test_graph_adjoint_identity():
    E = GRAPHS[3][1]
    q = E.shape[0]
    alg = _graph_alg(E, [2, 3, 1, 2, 2], [3, 1, 2, 2, 1])
    g = rng(45)
    M = 15
    X, W, G = g.standard_normal((M, alg.K)), g.standard_normal((alg.K, alg.N)), g.standard_normal((M, alg.N))
    t = g.integers(0, q, M).astype(np.int32)
    Y, _, _, _ = oracle.proj_fwd(alg, t, X, W)
    dX = oracle.proj_bwd_data(alg, t, G, W)
    dW, _ = oracle.proj_bwd_weight(alg, t, X, G)
    a, b, c = np.sum(Y * G), np.sum(X * dX), np.sum(W * dW)
    assert abs(a - b) < 1e-10 * max(1, abs(a)) and abs(a - c) < 1e-10 * max(1, abs(a))


# ---- P17: algebraic attention (appendix "Attention Extension") -------------------------

def _dense_causal_attention(Q, K, V, S, scale):
    """Textbook causal softmax attention of one head for one sequence."""
    s = (Q @ K.T) * scale
    s[np.triu_indices(S, 1)] = -np.inf
    s -= s.max(1, keepdims=True)
    P = np.exp(s)
    P /= P.sum(1, keepdims=True)
    return P @ V


def test_attention_dense_law_is_ordinary_attention():
    """With every group in the support the score is the standard
    <Q_p, K_u> / sqrt(d_h) and the oracle is ordinary causal attention."""
    q, m, S = 4, 8, 13
    g = rng(50)
    Q, K, V = (g.standard_normal((S, q * m)) for _ in range(3))
    pt = (np.arange(S) % q).astype(np.int32)
    O = oracle.attn_fwd(q, "dense", m, 1, 1, 1, S, pt, Q, K, V)
    np.testing.assert_allclose(O, _dense_causal_attention(Q, K, V, S, 1 / np.sqrt(q * m)), atol=1e-12)
    # q = 1 under the star law is the same ordinary attention with 1/sqrt(m)
    O1 = oracle.attn_fwd(1, "star", q * m, 1, 1, 1, S, np.zeros(S, np.int32), Q, K, V)
    np.testing.assert_allclose(O1, _dense_causal_attention(Q, K, V, S, 1 / np.sqrt(q * m)), atol=1e-12)


@pytest.mark.parametrize("law,q", [("star", 2), ("star", 3), ("tensor2", 4)])
def test_attention_raw_score_is_the_typed_product(law, q):
    """The raw score of a type-i query and a type-j key is the (query, key)
    entry of Q *_q K^T (the block identity stated with eq.
    attention-raw-score): computed here through the (pinned) projection
    oracle with X = Q and W = K^T, its output groups the keys of each type.
    The values are one-hot on the positions, so the output row of query p
    is its softmax row, whose log-ratios give the scores; those must equal
    the typed product divided by sqrt(|F(i,j)| m)."""
    m = 6
    S = q * m  # V_u = e_u needs d_h = q m >= S
    g = rng(51, q)
    Q, K = g.standard_normal((S, q * m)), g.standard_normal((S, q * m))
    V = np.eye(S)
    pt = np.array([(5 * p + 1) % q for p in range(S)], np.int32)  # a non-cyclic schedule
    O = oracle.attn_fwd(q, law, m, 1, 1, 1, S, pt, Q, K, V)
    order = np.argsort(pt, kind="stable")
    widths = tuple(int((pt == j).sum()) for j in range(q))
    alg = Alg(q, (m,) * q, widths, law)
    R, _, _, _ = oracle.proj_fwd(alg, pt, Q, K[order].T)
    raw = np.empty((S, S))
    raw[:, order] = R
    nf = np.array([[sum(oracle.attn_in_group(law, i, j, a) for a in range(q)) for j in range(q)] for i in range(q)])
    score = raw / np.sqrt(nf[pt][:, pt] * m)
    for p in range(1, S):
        lr = np.log(O[p, :p + 1]) - np.log(O[p, 0])
        np.testing.assert_allclose(lr, score[p, :p + 1] - score[p, 0], atol=1e-9)
        assert np.all(O[p, p + 1:] == 0)  # causal
    # star law: |F(i,i)| = 1 and |F(i,j)| = 2 (eq. attention-support-size)
    if law == "star":
        assert all(nf[i, i] == 1 for i in range(q))
        assert all(nf[i, j] == 2 for i in range(q) for j in range(q) if i != j)


def test_attention_causality_gqa_and_decode():
    """A query's output ignores later keys and values (Proposition
    "Causality"); head h reads key/value head h // (n_heads / n_kv); and one
    decode step over a cache of L positions is row L - 1 of the forward."""
    q, m, B, S, nh, nkv = 2, 8, 2, 11, 4, 2
    dh = q * m
    g = rng(52)
    Q = g.standard_normal((B * S, nh * dh))
    K = g.standard_normal((B * S, nkv * dh))
    V = g.standard_normal((B * S, nkv * dh))
    pt = (np.arange(S) % q).astype(np.int32)
    O = oracle.attn_fwd(q, "star", m, nh, nkv, B, S, pt, Q, K, V)
    K2, V2 = K.copy(), V.copy()
    K2[S + 7:2 * S] += 3.0
    V2[S + 7:2 * S] -= 5.0
    O2 = oracle.attn_fwd(q, "star", m, nh, nkv, B, S, pt, Q, K2, V2)
    np.testing.assert_array_equal(O2[:S + 7], O[:S + 7])
    assert not np.allclose(O2[S + 7:], O[S + 7:])
    for h in range(nh):
        hk = h // (nh // nkv)
        Oh = oracle.attn_fwd(q, "star", m, 1, 1, B, S, pt, Q[:, h * dh:(h + 1) * dh],
                             K[:, hk * dh:(hk + 1) * dh], V[:, hk * dh:(hk + 1) * dh])
        np.testing.assert_allclose(O[:, h * dh:(h + 1) * dh], Oh, atol=1e-13)
    L = np.array([5, 11], np.int32)
    Kc, Vc = K.reshape(B, S, -1), V.reshape(B, S, -1)
    Qd = np.stack([Q[b * S + L[b] - 1] for b in range(B)])
    Od = oracle.attn_decode(q, "star", m, nh, nkv, pt, L, Qd, Kc, Vc)
    for b in range(B):
        np.testing.assert_allclose(Od[b], O[b * S + L[b] - 1], atol=1e-13)


def test_attention_log_sum_exp():
    """The log of each query's softmax denominator: for the dense law it is
    scipy's logsumexp of the causal row of Q K^T / sqrt(d_h); for the star
    law, asking for it leaves the output unchanged, and at the first
    position (a single key of the query's own type) it is that key's score
    over the one group F(0, 0) = {0}."""
    from scipy.special import logsumexp
    q, m, S, nh = 4, 8, 17, 2
    dh = q * m
    g = rng(53)
    Q, K, V = g.standard_normal((S, nh * dh)), g.standard_normal((S, dh)), g.standard_normal((S, dh))
    pt = np.array([(3 * p + 2) % q for p in range(S)], np.int32)
    _, lse = oracle.attn_fwd(q, "dense", m, nh, 1, 1, S, pt, Q, K, V, want_lse=True)
    for h in range(nh):
        s = Q[:, h * dh:(h + 1) * dh] @ K.T / np.sqrt(dh)
        for p in range(S):
            np.testing.assert_allclose(lse[0, h, p], logsumexp(s[p, :p + 1]), rtol=0, atol=1e-12)
    m2, S2 = 6, 12
    Qs, Ks = g.standard_normal((S2, 2 * m2)), g.standard_normal((S2, 2 * m2))
    pt2 = (np.arange(S2) % 2).astype(np.int32)
    O, lse2 = oracle.attn_fwd(2, "star", m2, 1, 1, 1, S2, pt2, Qs, Ks, np.eye(S2), want_lse=True)
    np.testing.assert_allclose(O.sum(1), 1.0, atol=1e-13)
    O_plain = oracle.attn_fwd(2, "star", m2, 1, 1, 1, S2, pt2, Qs, Ks, np.eye(S2))
    np.testing.assert_array_equal(O, O_plain)
    # at p = 0 the single key gives lse = s_00 = <Q_0^(0), K_0^(0)> / sqrt(m)
    np.testing.assert_allclose(lse2[0, 0, 0], Qs[0, :m2] @ Ks[0, :m2] / np.sqrt(m2), atol=1e-13)
