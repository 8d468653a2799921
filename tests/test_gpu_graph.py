"""GPU parity for the graph algebra Q_G (law "graph", Sec. "Graph Products
with Exact Cost"): forward with bias and GELU, activation gradient with and
without the fused act', weight and bias gradients, an FFN training step and
the decode kernels, against the fp64 oracle on the same seeded inputs.

Under Q_G a type-i row reaches only its vertex slot and the edge slots of its
out-edges, so the checks include the output groups that are not slots of a
row (act(bias) forward, zero activation gradient), the input groups that are
never read, and the weight blocks of non-edges (zero gradient).  The graphs
mix sparse, dense and degenerate cases (an isolated vertex, a vertex with
every out-edge, a cycle); widths are unequal and rows span several tiles
with ragged tails.
"""

import numpy as np
import pytest

import oracle
import synth
from helpers import TOL_BF16, TOL_F32, f32_dev, rel_fro, to_dev, to_host, types_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    assert torch.cuda.is_available(), "GPU parity tests need a GPU"
    import paper_2609_32814_amd as P
    return P


def bar(dtype):
    return TOL_F32 if dtype == "f32" else TOL_BF16


def _graph(q, p, seed):
    g = np.random.default_rng([60, q, seed])
    E = (g.random((q, q)) < p).astype(np.uint8)
    np.fill_diagonal(E, 0)
    return E


GRAPHS = {
    "cycle3": np.array([[0, 1, 0], [0, 0, 1], [1, 0, 0]], np.uint8),
    # vertex 0 reaches everyone, vertex 3 is isolated
    "hub4": np.array([[0, 1, 1, 1], [0, 0, 1, 0], [0, 0, 0, 0], [0, 0, 0, 0]], np.uint8),
    "random6": _graph(6, 0.35, 1),
    "empty2": np.zeros((2, 2), np.uint8),
}

# (graph, s, r, M)
SHAPES = [
    ("cycle3", [128, 64, 192], [256, 128, 64], 700),
    ("hub4", [64, 128, 64, 192], [256, 64, 128, 64], 1100),
    ("random6", [64] * 6, [96, 64, 128, 64, 32, 64], 900),
    ("empty2", [128, 64], [192, 128], 333),
]


def algs(P, name, s, r):
    E = GRAPHS[name]
    q = E.shape[0]
    return P.Algebra(q, s, r, "graph", E), oracle.Alg(q, tuple(s), tuple(r), "graph", tuple(map(tuple, E)))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name,s,r,M", SHAPES)
def test_graph_fwd_parity(P, dtype, name, s, r, M):
    import torch
    ga, oa = algs(P, name, s, r)
    q = oa.q
    seed = 1600 + M
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, dtype)
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.05, dtype)
    b = synth.gaussian(seed, 2, (oa.N,), 0.1, "f32")
    t = np.random.default_rng([seed, 3]).integers(0, q, M).astype(np.int32)
    Y, Z = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), f32_dev(b.exact), "gelu", Z_out=True,
                           out_dtype=torch.float32)
    refY, refZ, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact, b.exact, "gelu", want_z=True)
    gY, gZ = to_host(Y), to_host(Z)
    assert rel_fro(gZ, refZ) <= bar(dtype)
    assert rel_fro(gY, refY) <= bar(dtype)
    # the output groups that are not slots of a row hold exactly bias / act(bias)
    R = np.concatenate([[0], np.cumsum(r)])
    E = GRAPHS[name]
    for b_ in range(0, M, 37):
        i = t[b_]
        for j in range(q):
            if j != i and not E[i, j]:
                np.testing.assert_array_equal(gZ[b_, R[j]:R[j + 1]], b.raw[R[j]:R[j + 1]].astype(np.float64))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("name,s,r,M", SHAPES)
def test_graph_bwd_data_parity(P, dtype, fused, name, s, r, M):
    import torch
    ga, oa = algs(P, name, s, r)
    seed = 1700 + M
    dY = synth.gaussian(seed, 0, (M, oa.N), 1.0, dtype)
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.05, dtype)
    Zp = synth.gaussian(seed, 2, (M, oa.K), 1.0, dtype) if fused else None
    t = np.random.default_rng([seed, 3]).integers(0, oa.q, M).astype(np.int32)
    dX = P.star_proj_bwd_data(ga, types_dev(t), to_dev(dY), to_dev(W), Z_prev=to_dev(Zp) if fused else None,
                              act_prev="gelu" if fused else "none", out_dtype=torch.float32)
    ref = oracle.proj_bwd_data(oa, t, dY.exact, W.exact, Zprev=Zp.exact if fused else None,
                               act_prev="gelu" if fused else "none")
    got = to_host(dX)
    assert rel_fro(got, ref) <= bar(dtype)
    # the input groups that are not slots get an exactly zero gradient
    assert np.all(got[ref == 0] == 0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name,s,r,M", SHAPES)
def test_graph_bwd_weight_parity(P, dtype, name, s, r, M):
    ga, oa = algs(P, name, s, r)
    seed = 1800 + M
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, dtype)
    dY = synth.gaussian(seed, 1, (M, oa.N), 1.0, dtype)
    t = np.random.default_rng([seed, 3]).integers(0, oa.q, M).astype(np.int32)
    dW, db = P.star_proj_bwd_weight(ga, types_dev(t), to_dev(X), to_dev(dY))
    rW, rb = oracle.proj_bwd_weight(oa, t, X.exact, dY.exact)
    gW = to_host(dW)
    assert rel_fro(gW, rW) <= bar(dtype)
    assert rel_fro(to_host(db), rb) <= bar(dtype)
    # the blocks of non-edges are not parameters: exactly zero
    assert np.all(gW[rW == 0] == 0)
    # deterministic: a second call is bitwise equal
    dW2, db2 = P.star_proj_bwd_weight(ga, types_dev(t), to_dev(X), to_dev(dY))
    import torch
    assert torch.equal(dW, dW2) and torch.equal(db, db2)


def test_graph_ffn_train_step_parity(P):
    """Up 768 -> 1536 and down 1536 -> 768 under one graph on q = 4 groups,
    one plan for all six products."""
    import torch
    E = GRAPHS["hub4"]
    q, D, F, M = 4, 768, 1536, 2048
    up_g, up_o = P.Algebra.equal(q, D, F, "graph", E), oracle.Alg.equal(q, D, F, "graph", E)
    dn_g, dn_o = P.Algebra.equal(q, F, D, "graph", E), oracle.Alg.equal(q, F, D, "graph", E)
    seed = 1900
    X = synth.gaussian(seed, 0, (M, D), 1.0, "bf16")
    Wu = synth.gaussian(seed, 1, (D, F), 0.03, "bf16")
    Wd = synth.gaussian(seed, 2, (F, D), 0.03, "bf16")
    bu = synth.gaussian(seed, 3, (F,), 0.02, "f32")
    bd = synth.gaussian(seed, 4, (D,), 0.02, "f32")
    dY = synth.gaussian(seed, 5, (M, D), 1.0, "bf16")
    t = synth.sequence_types(M, q, 512)
    td = types_dev(t)
    Z, H, Y = P.star_ffn_fwd(up_g, dn_g, td, to_dev(X), to_dev(Wu), f32_dev(bu.exact), to_dev(Wd),
                             f32_dev(bd.exact), "gelu", out_dtype=torch.float32)
    g = P.star_ffn_bwd(up_g, dn_g, td, to_dev(X), Z, H, to_dev(Wu), to_dev(Wd), to_dev(dY), "gelu")
    rZ, rH, rY = oracle.ffn_fwd(up_o, dn_o, t, X.exact, Wu.exact, bu.exact, Wd.exact, bd.exact)
    ref = oracle.ffn_bwd(up_o, dn_o, t, X.exact, rZ, rH, Wu.exact, Wd.exact, dY.exact)
    assert rel_fro(to_host(Y), rY) <= TOL_BF16
    for k in ("dX", "dW_up", "dW_down", "db_up", "db_down"):
        assert rel_fro(to_host(g[k]), ref[k]) <= TOL_BF16, k


@pytest.mark.parametrize("M,L", [(1, 3), (2, 3), (9, 3), (40, 2), (5, 33)])
def test_graph_decode_parity(P, M, L):
    """The decode kernels under the graph law: the resident stack (M <= 2),
    the counter stack and the per-projection kernel (33 layers)."""
    import torch
    E = GRAPHS["hub4"]
    q = 4
    D, F = (256, 512) if L < 33 else (128, 256)
    up_g, up_o = P.Algebra.equal(q, D, F, "graph", E), oracle.Alg.equal(q, D, F, "graph", E)
    dn_g, dn_o = P.Algebra.equal(q, F, D, "graph", E), oracle.Alg.equal(q, F, D, "graph", E)
    seed = 2000 + M + L
    Wu = [synth.gaussian(seed, 10 + l, (D, F), 0.05, "bf16") for l in range(L)]
    Wd = [synth.gaussian(seed, 100 + l, (F, D), 0.05, "bf16") for l in range(L)]
    bu = [synth.gaussian(seed, 200 + l, (F,), 0.02, "f32") for l in range(L)]
    bd = [synth.gaussian(seed, 300 + l, (D,), 0.02, "f32") for l in range(L)]
    X = synth.gaussian(seed, 1, (M, D), 1.0, "bf16")
    t = (synth.decode_positions(seed, M) % q).astype(np.int32)
    Y = P.star_decode(up_g, dn_g, types_dev(t), to_dev(X), [to_dev(w) for w in Wu],
                      [f32_dev(b.exact) for b in bu], [to_dev(w) for w in Wd],
                      [f32_dev(b.exact) for b in bd], "gelu", True, out_dtype=torch.float32)
    ref = oracle.decode_stack(up_o, dn_o, t, X.exact, [w.exact for w in Wu], [b.exact for b in bu],
                              [w.exact for w in Wd], [b.exact for b in bd])
    assert rel_fro(to_host(Y), ref) <= TOL_BF16


def test_graph_complete_equals_star(P):
    """The complete graph runs the star law's products: outputs agree with
    the star law's to rounding."""
    import torch
    q = 3
    E = np.ones((q, q), np.uint8)
    s, r, M = [64, 128, 64], [128, 64, 192], 777
    g_graph = P.Algebra(q, s, r, "graph", E)
    g_star = P.Algebra(q, s, r, "star")
    X = to_dev(synth.gaussian(2100, 0, (M, sum(s)), 1.0, "bf16"))
    W = to_dev(synth.gaussian(2100, 1, (sum(s), sum(r)), 0.05, "bf16"))
    t = types_dev(np.random.default_rng([2100, 3]).integers(0, q, M).astype(np.int32))
    a = P.star_proj_fwd(g_graph, t, X, W, out_dtype=torch.float32)
    b = P.star_proj_fwd(g_star, t, X, W, out_dtype=torch.float32)
    assert rel_fro(to_host(a), to_host(b)) <= 1e-6
