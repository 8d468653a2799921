"""GPU parity: the HIP path through the C ABI against the fp64 CPU oracle.

Every case draws its inputs from ``synth`` with a fixed seed, runs the same
values through both sides and compares element by element with the relative
Frobenius bar of the operand precision (``helpers.TOL_*``).  Small cases span
several 128 x 128 tiles with ragged tails; the full-size cases use the shapes
and launch configuration the benchmark times and compare sampled rows (the
projection is row-local) or sampled weight-gradient entries.
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


def algs(P, q, s, r, law="star"):
    return P.Algebra(q, s, r, law), oracle.Alg(q, tuple(s), tuple(r), law)


def bar(dtype):
    return TOL_F32 if dtype == "f32" else TOL_BF16


# ---- forward -------------------------------------------------------------------

def test_cfg1_fp32_q2(P):
    """64 x 128 rows of two 64-wide groups, W 128 x 128, N(0,1), t = b mod 2."""
    ga, oa = algs(P, 2, [64, 64], [64, 64])
    X = synth.gaussian(1, 0, (64, 128), 1.0, "f32")
    W = synth.gaussian(1, 1, (128, 128), 1.0, "f32")
    t = synth.cyclic_types(64, 2)
    Y = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W))
    ref, _, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact)
    assert rel_fro(to_host(Y), ref) <= TOL_F32
    # against the masked dense product too (independent formulation)
    gk = np.repeat([0, 1], 64)
    for i in (0, 1):
        rows = t == i
        mask = (gk[:, None] == i) | (gk[:, None] == gk[None, :])
        np.testing.assert_allclose(to_host(Y)[rows], X.exact[rows] @ (W.exact * mask),
                                   rtol=0, atol=1e-4)


@pytest.mark.parametrize("law", ["star", "dense"])
@pytest.mark.parametrize("dtype,out", [("f32", "f32"), ("bf16", "f32"), ("bf16", "bf16")])
@pytest.mark.parametrize("q,s,r,M,types", [
    (2, [64, 64], [64, 64], 64, "cyclic"),
    (2, [136, 120], [200, 56], 333, "cyclic"),
    (3, [64, 24, 104], [96, 160, 40], 517, "random"),
    (5, [16, 32, 8, 48, 24], [40, 8, 72, 16, 32], 700, "random"),
    (4, [32] * 4, [48] * 4, 300, "missing"),       # one type class is empty
    (8, [16] * 8, [32] * 8, 258, "offset"),
    (1, [72], [136], 130, "cyclic"),
])
def test_fwd_parity(P, law, dtype, out, q, s, r, M, types):
    import torch
    ga, oa = algs(P, q, s, r, law)
    seed = 100 + q
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, dtype)
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.05, dtype)
    bias = synth.gaussian(seed, 2, (oa.N,), 0.02, "f32")
    rng = np.random.default_rng([seed, 3])
    if types == "cyclic":
        t = synth.cyclic_types(M, q)
    elif types == "offset":
        t = synth.cyclic_types(M, q, offset=3)
    else:
        t = rng.integers(0, q, M).astype(np.int32)
        if types == "missing":
            t[t == 1] = 2
    odt = torch.float32 if out == "f32" else torch.bfloat16
    Y, Z = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), f32_dev(bias.exact), "gelu",
                           Z_out=True, out_dtype=odt)
    refY, refZ, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact, bias.exact, "gelu", want_z=True)
    tol = TOL_F32 if (dtype == "f32" and out == "f32") else TOL_BF16
    assert rel_fro(to_host(Z), refZ) <= tol
    assert rel_fro(to_host(Y), refY) <= tol


def test_fwd_one_row_of_each_type(P):
    ga, oa = algs(P, 4, [24, 40, 16, 48], [32, 8, 56, 24])
    for ty in range(4):
        t = np.array([ty], np.int32)
        X = synth.gaussian(7, ty, (1, oa.K), 1.0, "f32")
        W = synth.gaussian(7, 10, (oa.K, oa.N), 1.0, "f32")
        Y = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W))
        ref, _, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact)
        assert rel_fro(to_host(Y), ref) <= TOL_F32


def test_fwd_max_q(P):
    q = 64
    ga, oa = algs(P, q, [8] * q, [16] * q)
    M = 1000
    X = synth.gaussian(8, 0, (M, oa.K), 1.0, "bf16")
    W = synth.gaussian(8, 1, (oa.K, oa.N), 0.05, "bf16")
    t = synth.cyclic_types(M, q)
    import torch
    Y = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), out_dtype=torch.float32)
    ref, _, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact)
    assert rel_fro(to_host(Y), ref) <= TOL_BF16


def test_fwd_m0_is_noop(P):
    import torch
    ga, _ = algs(P, 2, [64, 64], [64, 64])
    Y = torch.full((0, 128), 7.0, device="cuda")
    X = torch.empty((0, 128), device="cuda")
    W = torch.zeros((128, 128), device="cuda")
    P.star_proj_fwd(ga, torch.empty(0, dtype=torch.int32, device="cuda"), X, W, Y=Y)
    torch.cuda.synchronize()


def test_out_of_range_types_left_out(P):
    import torch
    ga, oa = algs(P, 3, [32, 32, 64], [64, 32, 32])
    M = 200
    X = synth.gaussian(9, 0, (M, oa.K), 1.0, "f32")
    W = synth.gaussian(9, 1, (oa.K, oa.N), 1.0, "f32")
    t = synth.cyclic_types(M, 3)
    bad = np.array([5, 77, 150])
    t_bad = t.copy()
    t_bad[bad] = [3, -1, 9]
    td = types_dev(t_bad)
    assert P.star_validate_types(td, 3) == 3
    assert P.star_validate_types(types_dev(t), 3) == 0
    Y = torch.full((M, oa.N), 12345.0, device="cuda")
    P.star_proj_fwd(ga, td, to_dev(X), to_dev(W), Y=Y)
    got = to_host(Y)
    assert np.all(got[bad] == 12345.0)
    good = np.setdiff1d(np.arange(M), bad)
    ref, _, _, _ = oracle.proj_fwd(oa, t[good], X.exact[good], W.exact)
    assert rel_fro(got[good], ref) <= TOL_F32


# ---- bf16 shapes with every K group wider than 64 (the pipelined kernel) --------

PIPE_SHAPES = [
    # several row tiles per type with a ragged last one; K groups with tails
    # of 8..56 past a multiple of 64; output groups that end inside a tile
    (2, [200, 136], [328, 200], 1500, "cyclic"),
    (3, [72, 264, 96], [136, 72, 392], 2000, "random"),
    # long contractions (17 and 9 K steps) and a one-type class of 1 row
    (2, [1040, 520], [264, 136], 771, "one_row"),
    (1, [776], [392], 1100, "cyclic"),
    # groups 384 wide (whole 256 x 192 tiles) next to ones with a tail of 8
    (2, [384, 392], [384, 200], 2100, "random"),
]


def _types(kind, M, q, seed):
    rng = np.random.default_rng([seed, 3])
    if kind == "cyclic":
        return synth.cyclic_types(M, q)
    t = rng.integers(0, q, M).astype(np.int32)
    if kind == "one_row":
        t[:] = 0
        t[M // 2] = 1
    return t


@pytest.mark.parametrize("tiles", ["wide", "wide192", "small"])
@pytest.mark.parametrize("law", ["star", "dense"])
@pytest.mark.parametrize("out", ["f32", "bf16"])
@pytest.mark.parametrize("q,s,r,M,types", PIPE_SHAPES)
def test_fwd_pipelined_shapes(P, tiles, law, out, q, s, r, M, types):
    import torch
    ga, oa = algs(P, q, s, r, law)
    seed = 400 + q + M
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, "bf16")
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.03, "bf16")
    bias = synth.gaussian(seed, 2, (oa.N,), 0.02, "f32")
    t = _types(types, M, q, seed)
    odt = torch.float32 if out == "f32" else torch.bfloat16
    P.star_set_fwd_tiles(tiles)
    try:
        Y, Z = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), f32_dev(bias.exact), "gelu",
                               Z_out=True, out_dtype=odt)
    finally:
        P.star_set_fwd_tiles("auto")
    refY, refZ, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact, bias.exact, "gelu", want_z=True)
    assert rel_fro(to_host(Z), refZ) <= TOL_BF16
    assert rel_fro(to_host(Y), refY) <= TOL_BF16
    # every row individually (a dropped or duplicated tile shows up here)
    diff = np.linalg.norm(to_host(Z) - refZ, axis=1) / np.maximum(np.linalg.norm(refZ, axis=1), 1e-30)
    assert diff.max() <= 4 * TOL_BF16


@pytest.mark.parametrize("law", ["star", "dense"])
@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("q,s,r,M,types", PIPE_SHAPES)
def test_bwd_data_pipelined_shapes(P, law, fused, q, s, r, M, types):
    import torch
    ga, oa = algs(P, q, s, r, law)
    seed = 500 + q + M
    dY = synth.gaussian(seed, 0, (M, oa.N), 1.0, "bf16")
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.03, "bf16")
    Zp = synth.gaussian(seed, 2, (M, oa.K), 1.0, "bf16") if fused else None
    t = _types(types, M, q, seed)
    dX = P.star_proj_bwd_data(ga, types_dev(t), to_dev(dY), to_dev(W),
                              Z_prev=to_dev(Zp) if fused else None,
                              act_prev="gelu" if fused else "none", out_dtype=torch.float32)
    ref = oracle.proj_bwd_data(oa, t, dY.exact, W.exact, Zprev=Zp.exact if fused else None,
                               act_prev="gelu" if fused else "none")
    got = to_host(dX)
    assert rel_fro(got, ref) <= TOL_BF16
    diff = np.linalg.norm(got - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-30)
    assert diff.max() <= 4 * TOL_BF16


def test_pipelined_out_of_range_types_left_out(P):
    import torch
    ga, oa = algs(P, 2, [136, 200], [264, 72])
    M = 900
    X = synth.gaussian(13, 0, (M, oa.K), 1.0, "bf16")
    W = synth.gaussian(13, 1, (oa.K, oa.N), 0.03, "bf16")
    t = synth.cyclic_types(M, 2)
    bad = np.array([0, 255, 256, 899])
    t_bad = t.copy()
    t_bad[bad] = [2, -5, 7, 1000]
    Y = torch.full((M, oa.N), 12345.0, device="cuda")
    P.star_proj_fwd(ga, types_dev(t_bad), to_dev(X), to_dev(W), Y=Y)
    got = to_host(Y)
    assert np.all(got[bad] == 12345.0)
    good = np.setdiff1d(np.arange(M), bad)
    ref, _, _, _ = oracle.proj_fwd(oa, t[good], X.exact[good], W.exact)
    assert rel_fro(got[good], ref) <= TOL_BF16


# ---- backward -------------------------------------------------------------------

@pytest.mark.parametrize("law", ["star", "dense"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("q,s,r,M", [
    (2, [64, 64], [96, 160], 333),
    (3, [40, 64, 24], [48, 16, 136], 450),
    (4, [32] * 4, [64] * 4, 257),
])
@pytest.mark.parametrize("fused", [False, True])
def test_bwd_data_parity(P, law, dtype, q, s, r, M, fused):
    ga, oa = algs(P, q, s, r, law)
    seed = 200 + q
    dY = synth.gaussian(seed, 0, (M, oa.N), 1.0, dtype)
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.05, dtype)
    Zp = synth.gaussian(seed, 2, (M, oa.K), 1.0, dtype) if fused else None
    t = np.random.default_rng([seed, 3]).integers(0, q, M).astype(np.int32)
    import torch
    dX = P.star_proj_bwd_data(ga, types_dev(t), to_dev(dY), to_dev(W),
                              Z_prev=to_dev(Zp) if fused else None,
                              act_prev="gelu" if fused else "none", out_dtype=torch.float32)
    ref = oracle.proj_bwd_data(oa, t, dY.exact, W.exact, Zprev=Zp.exact if fused else None,
                               act_prev="gelu" if fused else "none")
    assert rel_fro(to_host(dX), ref) <= bar(dtype)


@pytest.mark.parametrize("law", ["star", "tensor2"])
@pytest.mark.parametrize("mode", ["fwd", "bwd_data"])
def test_half_height_last_round(P, law, mode):
    """Shapes whose first pass of tiles fits in one round of the persistent
    grid (256 workgroups) while whole tiles would deal out unevenly: with the
    star law the second pass then runs in half-height tiles (128 of 256 rows;
    the waves of the empty half skip their MFMAs and epilogue) dealt to the
    workgroups without a first-pass tile first.  Every output against the
    oracle; the type counts are not multiples of 128, so the last half tile
    of each class is ragged.  (fwd: 2 x 13 row tiles x 8 column tiles per
    pass; activation gradient: 2 x 24 row tiles x 4 column tiles per pass.
    The tensor-square law runs the same shapes in whole tiles.)"""
    import torch
    q = 2 if law == "star" else 4
    if mode == "fwd":
        s, r, M = [256 // q] * q, [4096 // q] * q, 6181
    else:
        s, r, M = [2048 // q] * q, [256 // q] * q, 12037
    ga, oa = algs(P, q, s, r, law)
    seed = 400 + q
    t = synth.cyclic_types(M, q)
    if mode == "fwd":
        X = synth.gaussian(seed, 0, (M, oa.K), 1.0, "bf16")
        W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.05, "bf16")
        bias = synth.gaussian(seed, 2, (oa.N,), 0.02, "f32")
        Y, Z = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), f32_dev(bias.exact), "gelu",
                               Z_out=True)
        refY, refZ, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact, bias.exact, "gelu", want_z=True)
        assert rel_fro(to_host(Z), refZ) <= TOL_BF16
        assert rel_fro(to_host(Y), refY) <= TOL_BF16
    else:
        dY = synth.gaussian(seed, 0, (M, oa.N), 1.0, "bf16")
        W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.05, "bf16")
        Zp = synth.gaussian(seed, 2, (M, oa.K), 1.0, "bf16")
        dX = P.star_proj_bwd_data(ga, types_dev(t), to_dev(dY), to_dev(W), Z_prev=to_dev(Zp),
                                  act_prev="gelu", out_dtype=torch.float32)
        ref = oracle.proj_bwd_data(oa, t, dY.exact, W.exact, Zprev=Zp.exact, act_prev="gelu")
        assert rel_fro(to_host(dX), ref) <= TOL_BF16


@pytest.mark.parametrize("law", ["star", "dense"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("q,s,r,M", [
    (2, [64, 64], [96, 160], 333),      # one split
    (3, [40, 64, 24], [48, 16, 136], 4100),  # several splits, ragged
    (4, [32] * 4, [64] * 4, 2049),
    (2, [128, 128], [128, 128], 0),     # empty batch: zero gradients
    (2, [384, 392], [384, 384], 3000),  # output groups 384 wide
    (2, [384, 384], [512, 256], 2500),  # input groups 384 wide (192-row tiles)
])
def test_bwd_weight_parity(P, law, dtype, q, s, r, M):
    ga, oa = algs(P, q, s, r, law)
    seed = 300 + q
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, dtype)
    dY = synth.gaussian(seed, 1, (M, oa.N), 1.0, dtype)
    t = np.random.default_rng([seed, 3]).integers(0, q, M).astype(np.int32)
    dW, db = P.star_proj_bwd_weight(ga, types_dev(t), to_dev(X), to_dev(dY))
    rW, rb = oracle.proj_bwd_weight(oa, t, X.exact, dY.exact)
    if M == 0:
        assert np.all(to_host(dW) == 0) and np.all(to_host(db) == 0)
        return
    assert rel_fro(to_host(dW), rW) <= bar(dtype)
    assert rel_fro(to_host(db), rb) <= bar(dtype)
    # bitwise reproducible
    dW2, db2 = P.star_proj_bwd_weight(ga, types_dev(t), to_dev(X), to_dev(dY))
    assert np.array_equal(to_host(dW2), to_host(dW)) and np.array_equal(to_host(db2), to_host(db))


@pytest.mark.parametrize("r", [[384, 392], [1024, 1032]])
def test_bwd_weight_out_of_range_types_left_out(P, r):
    """Rows whose type is outside [0, q) are left out of the weight and bias
    gradients: the result equals the oracle's over the valid rows alone.  The
    bias column sums then walk the rows in type-sorted order through perm
    (the 16-row-lane blocks for 776 columns, the 8-row-lane ones for 2056)."""
    ga, oa = algs(P, 2, [384, 384], r)
    M = 3000
    X = synth.gaussian(331, 0, (M, oa.K), 1.0, "bf16")
    dY = synth.gaussian(331, 1, (M, oa.N), 1.0, "bf16")
    rng = np.random.default_rng([331, 3])
    t = rng.integers(0, 2, M).astype(np.int32)
    bad = rng.choice(M, size=M // 17, replace=False)
    t_bad = t.copy()
    t_bad[bad] = rng.choice(np.array([-1, 2, 7, 1 << 20], dtype=np.int32), size=bad.size)
    dW, db = P.star_proj_bwd_weight(ga, types_dev(t_bad), to_dev(X), to_dev(dY))
    good = np.setdiff1d(np.arange(M), bad)
    rW, rb = oracle.proj_bwd_weight(oa, t[good], X.exact[good], dY.exact[good])
    assert rel_fro(to_host(dW), rW) <= TOL_BF16
    assert rel_fro(to_host(db), rb) <= TOL_BF16


def test_bwd_weight_absent_type_gives_zero_blocks(P):
    ga, oa = algs(P, 3, [32, 48, 40], [56, 24, 64])
    M = 600
    X = synth.gaussian(11, 0, (M, oa.K), 1.0, "bf16")
    dY = synth.gaussian(11, 1, (M, oa.N), 1.0, "bf16")
    t = synth.cyclic_types(M, 3)
    t[t == 1] = 0
    dW, _ = P.star_proj_bwd_weight(ga, types_dev(t), to_dev(X), to_dev(dY))
    g = to_host(dW)
    # row block of group 1 (rows 32..80), off-diagonal columns: exactly zero
    assert np.all(g[32:80, :56] == 0) and np.all(g[32:80, 80:] == 0)
    rW, _ = oracle.proj_bwd_weight(oa, t, X.exact, dY.exact)
    assert rel_fro(g, rW) <= TOL_BF16


# ---- FFN forward + backward ----------------------------------------------------------

@pytest.mark.parametrize("q,D,F,M", [(2, 256, 1024, 1000), (4, 128, 512, 777)])
def test_ffn_train_step_parity(P, q, D, F, M):
    import torch
    up_g, up_o = algs(P, q, [D // q] * q, [F // q] * q)
    dn_g, dn_o = algs(P, q, [F // q] * q, [D // q] * q)
    seed = 400 + q
    X = synth.gaussian(seed, 0, (M, D), 1.0, "bf16")
    Wu = synth.gaussian(seed, 1, (D, F), 0.02, "bf16")
    Wd = synth.gaussian(seed, 2, (F, D), 0.02, "bf16")
    bu = synth.gaussian(seed, 3, (F,), 0.02, "f32")
    bd = synth.gaussian(seed, 4, (D,), 0.02, "f32")
    dY = synth.gaussian(seed, 5, (M, D), 1.0, "bf16")
    t = synth.sequence_types(M, q, 256)
    td = types_dev(t)
    Z, H, Y = P.star_ffn_fwd(up_g, dn_g, td, to_dev(X), to_dev(Wu), f32_dev(bu.exact), to_dev(Wd),
                             f32_dev(bd.exact), "gelu", out_dtype=torch.float32)
    rZ, rH, rY = oracle.ffn_fwd(up_o, dn_o, t, X.exact, Wu.exact, bu.exact, Wd.exact, bd.exact)
    assert rel_fro(to_host(Z), rZ) <= TOL_BF16
    assert rel_fro(to_host(H), rH) <= TOL_BF16
    assert rel_fro(to_host(Y), rY) <= TOL_BF16
    g = P.star_ffn_bwd(up_g, dn_g, td, to_dev(X), Z, H, to_dev(Wu), to_dev(Wd), to_dev(dY), "gelu")
    # the oracle's backward consumes its own forward's stored tensors
    ref = oracle.ffn_bwd(up_o, dn_o, t, X.exact, rZ, rH, Wu.exact, Wd.exact, dY.exact)
    for k in ("dZ", "dX", "dW_up", "db_up", "dW_down", "db_down"):
        assert rel_fro(to_host(g[k]), ref[k]) <= TOL_BF16, k


# ---- decode -------------------------------------------------------------------------

@pytest.mark.parametrize("M", [1, 2, 8, 12, 20, 32, 64])
@pytest.mark.parametrize("D,F,L", [(256, 1024, 1), (256, 1024, 3), (768, 3072, 12)])
def test_decode_parity(P, M, D, F, L):
    import torch
    up_g, up_o = algs(P, 2, [D // 2] * 2, [F // 2] * 2)
    dn_g, dn_o = algs(P, 2, [F // 2] * 2, [D // 2] * 2)
    seed = 500 + L
    Wu = [synth.gaussian(seed, 10 + l, (D, F), 0.02, "bf16") for l in range(L)]
    Wd = [synth.gaussian(seed, 40 + l, (F, D), 0.02, "bf16") for l in range(L)]
    bu = [synth.gaussian(seed, 70 + l, (F,), 0.02, "f32") for l in range(L)]
    bd = [synth.gaussian(seed, 100 + l, (D,), 0.02, "f32") for l in range(L)]
    X = synth.gaussian(seed, 1, (M, D), 1.0, "bf16")
    t = (synth.decode_positions(seed, M) % 2).astype(np.int32)
    Y = P.star_decode(up_g, dn_g, types_dev(t), to_dev(X), [to_dev(w) for w in Wu],
                      [f32_dev(b.exact) for b in bu], [to_dev(w) for w in Wd],
                      [f32_dev(b.exact) for b in bd], "gelu", True, out_dtype=torch.float32)
    ref = oracle.decode_stack(up_o, dn_o, t, X.exact, [w.exact for w in Wu], [b.exact for b in bu],
                              [w.exact for w in Wd], [b.exact for b in bd])
    assert rel_fro(to_host(Y), ref) <= TOL_BF16
    # the same step again gives bitwise the same result (counters reset)
    Y2 = P.star_decode(up_g, dn_g, types_dev(t), to_dev(X), [to_dev(w) for w in Wu],
                       [f32_dev(b.exact) for b in bu], [to_dev(w) for w in Wd],
                       [f32_dev(b.exact) for b in bd], "gelu", True, out_dtype=torch.float32)
    assert torch.equal(Y, Y2)


@pytest.mark.parametrize("M", [1, 2])
def test_decode_few_rows_more_up_tiles_than_down_items(P, M):
    """D = 24 + 24, F = 200 + 200: 26 up tiles of 16 columns but only 4 down
    tiles x 4 chunks of 128, so some workgroups own no down item and the
    stack must not keep the running state resident (its double-buffered
    partials rely on every workgroup reading them before writing its own);
    it runs the counter hand-offs instead, and must match the oracle over
    several layers and give the same bits twice."""
    import torch
    sD, sF = [24, 24], [200, 200]
    up_g, up_o = algs(P, 2, sD, sF)
    dn_g, dn_o = algs(P, 2, sF, sD)
    D, F, L = sum(sD), sum(sF), 4
    seed = 900 + M
    Wu = [synth.gaussian(seed, 10 + l, (D, F), 0.05, "bf16") for l in range(L)]
    Wd = [synth.gaussian(seed, 40 + l, (F, D), 0.05, "bf16") for l in range(L)]
    bu = [synth.gaussian(seed, 70 + l, (F,), 0.02, "f32") for l in range(L)]
    bd = [synth.gaussian(seed, 100 + l, (D,), 0.02, "f32") for l in range(L)]
    X = synth.gaussian(seed, 1, (M, D), 1.0, "bf16")
    t = (np.arange(M) % 2).astype(np.int32)

    def run():
        return P.star_decode(up_g, dn_g, types_dev(t), to_dev(X), [to_dev(w) for w in Wu],
                             [f32_dev(b.exact) for b in bu], [to_dev(w) for w in Wd],
                             [f32_dev(b.exact) for b in bd], "gelu", True, out_dtype=torch.float32)

    Y = run()
    ref = oracle.decode_stack(up_o, dn_o, t, X.exact, [w.exact for w in Wu], [b.exact for b in bu],
                              [w.exact for w in Wd], [b.exact for b in bd])
    assert rel_fro(to_host(Y), ref) <= TOL_BF16
    assert torch.equal(Y, run())


def test_decode_one_type_only_skips_blocks(P):
    """M = 1 of type 0: only the diagonal blocks and row block 0 are read;
    the result still matches the oracle (skipped chunks contribute nothing)."""
    import torch
    D, F = 256, 512
    up_g, up_o = algs(P, 2, [D // 2] * 2, [F // 2] * 2)
    dn_g, dn_o = algs(P, 2, [F // 2] * 2, [D // 2] * 2)
    Wu = synth.gaussian(600, 1, (D, F), 0.05, "bf16")
    Wd = synth.gaussian(600, 2, (F, D), 0.05, "bf16")
    X = synth.gaussian(600, 3, (1, D), 1.0, "bf16")
    for ty in (0, 1):
        t = np.array([ty], np.int32)
        Y = P.star_decode(up_g, dn_g, types_dev(t), to_dev(X), [to_dev(Wu)], None, [to_dev(Wd)],
                          None, "gelu", False, out_dtype=torch.float32)
        ref = oracle.decode_stack(up_o, dn_o, t, X.exact, [Wu.exact], [np.zeros(F)], [Wd.exact],
                                  [np.zeros(D)], residual=False)
        assert rel_fro(to_host(Y), ref) <= TOL_BF16


@pytest.mark.parametrize("path", ["stack_resident", "stack", "per_projection"])
def test_decode_out_of_range_types(P, path):
    """A row whose type lies outside [0, q) has an empty support in decode:
    every layer adds only b_down, so its Y row is X + the sum of the b_down[l]
    (fp32, in layer order); the other rows match the oracle run on them alone,
    and the step's status flag is clear.  The three decode kernels: the
    resident stack (M <= 2), the counter stack, the per-projection kernel
    (33 layers: more than the stack holds)."""
    import torch
    q = 2
    if path == "stack_resident":
        D, F, L, t = 256, 512, 3, np.array([1, 7], np.int32)
    elif path == "stack":
        D, F, L, t = 256, 512, 3, np.array([0, 1, 5, -1, 1, 0, 2, 0, 1], np.int32)
    else:
        D, F, L, t = 128, 256, 33, np.array([0, 1, 5, -1, 1], np.int32)
    M = t.size
    up_g, up_o = algs(P, q, [D // 2] * 2, [F // 2] * 2)
    dn_g, dn_o = algs(P, q, [F // 2] * 2, [D // 2] * 2)
    seed = 1400 + M
    Wu = [synth.gaussian(seed, 10 + l, (D, F), 0.05, "bf16") for l in range(L)]
    Wd = [synth.gaussian(seed, 100 + l, (F, D), 0.05, "bf16") for l in range(L)]
    bu = [synth.gaussian(seed, 200 + l, (F,), 0.02, "f32") for l in range(L)]
    bd = [synth.gaussian(seed, 300 + l, (D,), 0.02, "f32") for l in range(L)]
    X = synth.gaussian(seed, 1, (M, D), 1.0, "bf16")
    ws = torch.empty(P.star_workspace_bytes("decode", up_g, dn_g, M), dtype=torch.uint8, device="cuda")
    Y = P.star_decode(up_g, dn_g, types_dev(t), to_dev(X), [to_dev(w) for w in Wu],
                      [f32_dev(b.exact) for b in bu], [to_dev(w) for w in Wd],
                      [f32_dev(b.exact) for b in bd], "gelu", True, out_dtype=torch.float32, ws=ws)
    assert not P.star_decode_status(ws)
    got = to_host(Y)
    ok = (t >= 0) & (t < q)
    ref = oracle.decode_stack(up_o, dn_o, t[ok], X.exact[ok], [w.exact for w in Wu], [b.exact for b in bu],
                              [w.exact for w in Wd], [b.exact for b in bd])
    assert rel_fro(got[ok], ref) <= TOL_BF16
    h = X.exact[~ok].astype(np.float32)
    for b in bd:
        h = (h + b.exact.astype(np.float32)).astype(np.float32)
    np.testing.assert_allclose(got[~ok], h.astype(np.float64), rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("law", ["star", "dense"])
@pytest.mark.parametrize("M", [5, 40])
def test_decode_unequal_groups_q3(P, law, M):
    """q = 3 with unequal widths (D = 128 + 64 + 192, F = 256 + 128 + 384),
    random types: output tiles end inside 16-column tiles and K slices
    straddle group boundaries."""
    import torch
    sD, sF = [128, 64, 192], [256, 128, 384]
    up_g, up_o = algs(P, 3, sD, sF, law)
    dn_g, dn_o = algs(P, 3, sF, sD, law)
    D, F, L = sum(sD), sum(sF), 2
    seed = 700 + M
    Wu = [synth.gaussian(seed, 10 + l, (D, F), 0.03, "bf16") for l in range(L)]
    Wd = [synth.gaussian(seed, 40 + l, (F, D), 0.03, "bf16") for l in range(L)]
    bu = [synth.gaussian(seed, 70 + l, (F,), 0.02, "f32") for l in range(L)]
    bd = [synth.gaussian(seed, 100 + l, (D,), 0.02, "f32") for l in range(L)]
    X = synth.gaussian(seed, 1, (M, D), 1.0, "bf16")
    t = np.random.default_rng([seed, 5]).integers(0, 3, M).astype(np.int32)
    Y = P.star_decode(up_g, dn_g, types_dev(t), to_dev(X), [to_dev(w) for w in Wu],
                      [f32_dev(b.exact) for b in bu], [to_dev(w) for w in Wd],
                      [f32_dev(b.exact) for b in bd], "gelu", True, out_dtype=torch.bfloat16)
    ref = oracle.decode_stack(up_o, dn_o, t, X.exact, [w.exact for w in Wu], [b.exact for b in bu],
                              [w.exact for w in Wd], [b.exact for b in bd])
    # bf16 output against the oracle's result rounded the same way
    assert rel_fro(to_host(Y), oracle.round_bf16(ref)) <= TOL_BF16


@pytest.mark.parametrize("M", [8, 64])
def test_decode_wide_model(P, M):
    """D = 1024, F = 2048: at M = 64 the inputs no longer fit next to two
    weight slots in LDS and the stack runs one kernel per projection; at
    M = 8 it runs as one launch.  Both must match the oracle."""
    import torch
    D, F, L = 1024, 2048, 2
    up_g, up_o = algs(P, 2, [D // 2] * 2, [F // 2] * 2)
    dn_g, dn_o = algs(P, 2, [F // 2] * 2, [D // 2] * 2)
    seed = 800 + M
    Wu = [synth.gaussian(seed, 10 + l, (D, F), 0.02, "bf16") for l in range(L)]
    Wd = [synth.gaussian(seed, 40 + l, (F, D), 0.02, "bf16") for l in range(L)]
    X = synth.gaussian(seed, 1, (M, D), 1.0, "bf16")
    t = (synth.decode_positions(seed, M) % 2).astype(np.int32)
    Y = P.star_decode(up_g, dn_g, types_dev(t), to_dev(X), [to_dev(w) for w in Wu], None,
                      [to_dev(w) for w in Wd], None, "gelu", True, out_dtype=torch.float32)
    ref = oracle.decode_stack(up_o, dn_o, t, X.exact, [w.exact for w in Wu], [np.zeros(F)] * L,
                              [w.exact for w in Wd], [np.zeros(D)] * L)
    assert rel_fro(to_host(Y), ref) <= TOL_BF16


@pytest.mark.parametrize("M", [1, 16])
@pytest.mark.parametrize("D,F", [(1024, 8192), (6144, 2048)])
def test_decode_wider_than_4096(P, M, D, F):
    """A projection input wider than 4096 (the down map's F, or the up map's
    D): the per-projection kernel streams its weight slices through LDS in
    passes of 128 slices."""
    import torch
    q, L = 4, 2
    up_g, up_o = algs(P, q, [D // q] * q, [F // q] * q)
    dn_g, dn_o = algs(P, q, [F // q] * q, [D // q] * q)
    seed = 850 + M + D
    Wu = [synth.gaussian(seed, 10 + l, (D, F), 0.02, "bf16") for l in range(L)]
    Wd = [synth.gaussian(seed, 40 + l, (F, D), 0.02, "bf16") for l in range(L)]
    bu = [synth.gaussian(seed, 70 + l, (F,), 0.02, "f32") for l in range(L)]
    bd = [synth.gaussian(seed, 90 + l, (D,), 0.02, "f32") for l in range(L)]
    X = synth.gaussian(seed, 1, (M, D), 1.0, "bf16")
    t = (synth.decode_positions(seed, M) % q).astype(np.int32)
    Y = P.star_decode(up_g, dn_g, types_dev(t), to_dev(X), [to_dev(w) for w in Wu], [f32_dev(b.exact) for b in bu],
                      [to_dev(w) for w in Wd], [f32_dev(b.exact) for b in bd], "gelu", True,
                      out_dtype=torch.float32)
    ref = oracle.decode_stack(up_o, dn_o, t, X.exact, [w.exact for w in Wu], [b.exact for b in bu],
                              [w.exact for w in Wd], [b.exact for b in bd])
    assert rel_fro(to_host(Y), ref) <= TOL_BF16


# ---- full-size workloads (sampled) ---------------------------------------------------

def _sample_rows(M, n, seed):
    rng = np.random.default_rng([seed, 999])
    rows = np.unique(np.concatenate([[0, 1, M - 2, M - 1], rng.choice(M, n, replace=False)]))
    return rows


@pytest.mark.parametrize("law", ["star", "dense"])
def test_cfg2_full_size_sampled(P, law):
    """M = 8192 (8 x 1024), 768 -> 3072 in blocks 384 x 1536, bias + GELU,
    bf16 in / fp32 accumulate / bf16 out, t = position-in-sequence mod 2."""
    M, K, N = 8192, 768, 3072
    ga, oa = algs(P, 2, [384, 384], [1536, 1536], law)
    X = synth.gaussian(2, 0, (M, K), 1.0, "bf16")
    W = synth.gaussian(2, 1, (K, N), 0.02, "bf16")
    b = synth.gaussian(2, 2, (N,), 0.02, "f32")
    t = synth.sequence_types(M, 2, 1024)
    Y = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), f32_dev(b.exact), "gelu")
    rows = _sample_rows(M, 300, 2)
    ref, _, _, _ = oracle.proj_fwd(oa, t[rows], X.exact[rows], W.exact, b.exact, "gelu")
    assert rel_fro(to_host(Y[rows]), ref) <= TOL_BF16


@pytest.mark.parametrize("q", [2, 4, 8, 16])
def test_cfg4_qsweep_full_size_sampled(P, q):
    """Square star_q projection, block 256, d = 256 q, M = 16384, t = b mod q."""
    import torch
    M, d = 16384, 256 * q
    ga, oa = algs(P, q, [256] * q, [256] * q)
    X = synth.gaussian(4, q, (M, d), 1.0, "bf16")
    W = synth.gaussian(4, 100 + q, (d, d), (1.0 / d) ** 0.5, "bf16")
    t = synth.cyclic_types(M, q)
    Y = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W))
    rows = _sample_rows(M, 256, 4 + q)
    ref, _, macs, ppt = oracle.proj_fwd(oa, t[rows], X.exact[rows], W.exact)
    assert rel_fro(to_host(Y[rows]), ref) <= TOL_BF16
    # retained block products: 2q - 1 per type, vs q^2 for the dense law
    assert P.star_count_products(ga) == [2 * q - 1] * q == list(ppt)
    assert P.star_count_products(ga.with_law("dense")) == [q * q] * q
    assert P.star_count_macs(ga, np.bincount(t, minlength=q)) * q * q == (2 * q - 1) * M * d * d
    del Y
    torch.cuda.empty_cache()


def test_cfg3_full_size_sampled(P):
    """Training shapes: M = 16384 (16 x 1024), up 768 -> 3072 GELU, down 3072 -> 768.
    Forward and activation gradients on sampled rows (row-local); weight
    gradients on sampled entries of the full-batch sum."""
    import torch
    M, D, F = 16384, 768, 3072
    up_g, up_o = algs(P, 2, [384, 384], [1536, 1536])
    dn_g, dn_o = algs(P, 2, [1536, 1536], [384, 384])
    X = synth.gaussian(3, 0, (M, D), 1.0, "bf16")
    Wu = synth.gaussian(3, 1, (D, F), 0.02, "bf16")
    Wd = synth.gaussian(3, 2, (F, D), 0.02, "bf16")
    bu = synth.gaussian(3, 3, (F,), 0.02, "f32")
    bd = synth.gaussian(3, 4, (D,), 0.02, "f32")
    dY = synth.gaussian(3, 5, (M, D), 1.0, "bf16")
    t = synth.sequence_types(M, 2, 1024)
    td = types_dev(t)
    Xd, Wud, Wdd, dYd = to_dev(X), to_dev(Wu), to_dev(Wd), to_dev(dY)
    Z, H, Y = P.star_ffn_fwd(up_g, dn_g, td, Xd, Wud, f32_dev(bu.exact), Wdd, f32_dev(bd.exact),
                             "gelu")
    g = P.star_ffn_bwd(up_g, dn_g, td, Xd, Z, H, Wud, Wdd, dYd, "gelu")
    rows = _sample_rows(M, 200, 3)
    rZ, rH, rY = oracle.ffn_fwd(up_o, dn_o, t[rows], X.exact[rows], Wu.exact, bu.exact, Wd.exact,
                                bd.exact)
    assert rel_fro(to_host(Y[rows]), rY) <= TOL_BF16
    rg = oracle.ffn_bwd(up_o, dn_o, t[rows], X.exact[rows], rZ, rH, Wu.exact, Wd.exact,
                        dY.exact[rows])
    assert rel_fro(to_host(g["dZ"][rows]), rg["dZ"]) <= TOL_BF16
    assert rel_fro(to_host(g["dX"][rows]), rg["dX"]) <= TOL_BF16
    # weight gradients at full size on sampled entries, from the GPU's own
    # stored H and dZ would make the oracle depend on the HIP path, so check
    # the weight-gradient kernel at the same shapes on synthetic operands
    rng = np.random.default_rng([3, 77])
    for alg_g, alg_o, A_id, B_id, K_, N_ in ((up_g, up_o, 10, 11, D, F), (dn_g, dn_o, 12, 13, F, D)):
        A = synth.gaussian(3, A_id, (M, K_), 1.0, "bf16")
        B = synth.gaussian(3, B_id, (M, N_), 1.0, "bf16")
        dW, db = P.star_proj_bwd_weight(alg_g, td, to_dev(A), to_dev(B))
        kk = rng.integers(0, K_, 2048)
        nn = rng.integers(0, N_, 2048)
        ref = oracle.bwd_weight_entries(alg_o, t, A.exact, B.exact, kk, nn)
        assert rel_fro(to_host(dW)[kk, nn], ref) <= TOL_BF16
        assert rel_fro(to_host(db), B.exact.sum(0)) <= TOL_BF16
    torch.cuda.empty_cache()


def test_planned_entry_points_match(P):
    """A plan built once and reused gives the same bits as the plain calls."""
    import torch
    ga, oa = algs(P, 3, [64, 32, 32], [96, 64, 32])
    M = 700
    X = to_dev(synth.gaussian(12, 0, (M, oa.K), 1.0, "bf16"))
    W = to_dev(synth.gaussian(12, 1, (oa.K, oa.N), 0.05, "bf16"))
    dY = to_dev(synth.gaussian(12, 2, (M, oa.N), 1.0, "bf16"))
    t = types_dev(np.random.default_rng([12, 3]).integers(0, 3, M).astype(np.int32))
    plan = P.star_type_plan(3, t)
    assert torch.equal(P.star_proj_fwd(ga, t, X, W, act="gelu"),
                       P.star_proj_fwd_planned(ga, plan, X, W, act="gelu"))
    assert torch.equal(P.star_proj_bwd_data(ga, t, dY, W), P.star_proj_bwd_data_planned(ga, plan, dY, W))
    a, b = P.star_proj_bwd_weight(ga, t, X, dY)
    c, d = P.star_proj_bwd_weight_planned(ga, plan, X, dY)
    assert torch.equal(a, c) and torch.equal(b, d)


@pytest.mark.gpu
@pytest.mark.parametrize("q,M,bad", [(2, 8192, False), (1, 300, False), (3, 1000, True),
                                     (64, 5000, True), (7, 70001, True), (16, 64, False),
                                     (4, 16384, True), (2, 65536, True), (5, 65537, False),
                                     (3, 1025, True), (2, 1, False), (64, 65535, True),
                                     (8, 9000, True), (4, 3073, False), (1, 4096, True)])
def test_type_plan_is_stable_partition(P, q, M, bad):
    """The plan is the stable partition of the rows by type (a stable sort of
    the type keys, out-of-range types as a last key) and the per-type
    starts; checked element by element against numpy's stable sort."""
    import torch
    rng = np.random.default_rng([11, q, M])
    t = rng.integers(0, q, size=M).astype(np.int32)
    if bad:
        idx = rng.choice(M, size=max(1, M // 17), replace=False)
        t[idx] = rng.choice(np.array([-3, q, q + 5, 1 << 20], dtype=np.int32), size=idx.size)
    plan = P.star_type_plan(q, types_dev(t)).cpu().numpy()
    perm = plan[:4 * M].view(np.int32)
    off0 = (4 * M + 255) // 256 * 256
    offsets = plan[off0:off0 + 4 * (q + 1)].view(np.int32)
    key = np.where((t >= 0) & (t < q), t, q)
    np.testing.assert_array_equal(perm, np.argsort(key, kind="stable"))
    np.testing.assert_array_equal(offsets, [(key < i).sum() for i in range(q + 1)])


@pytest.mark.gpu
def test_graph_replay_matches_eager(P):
    """The type plan and the fused forward GEMM captured in one HIP graph give
    the eager result on every replay, with other eager work and
    synchronisations between the replays (the plan's scan and the GEMM's
    tile walk must not keep state across launches)."""
    import torch
    q, s, r, M = 2, 384, 1536, 2048
    ga = P.Algebra.equal(q, 2 * s, 2 * r)
    X = to_dev(synth.gaussian(9, 0, (M, 2 * s), 1.0, "bf16"))
    W = to_dev(synth.gaussian(9, 1, (2 * s, 2 * r), 0.02, "bf16"))
    b = f32_dev(synth.gaussian(9, 2, (2 * r,), 0.02, "f32").raw)
    t = types_dev(synth.sequence_types(M, q, 512))
    plan = torch.empty(P.star_plan_bytes(q, M), dtype=torch.uint8, device="cuda")
    Y = torch.empty((M, 2 * r), dtype=torch.bfloat16, device="cuda")
    P.star_type_plan(q, t, plan)
    ref = P.star_proj_fwd_planned(ga, plan, X, W, b, "gelu").clone()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        P.star_type_plan(q, t, plan)
        P.star_proj_fwd_planned(ga, plan, X, W, b, "gelu", Y=Y)
    other = P.Algebra.equal(4, 256, 512)
    for rep in range(4):
        Y.zero_()
        plan.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y, ref), f"replay {rep}"
        # eager work in between, on the same buffers' neighbours
        Xo = torch.randn(300, 256, device="cuda").to(torch.bfloat16)
        Wo = torch.randn(256, 512, device="cuda").to(torch.bfloat16)
        P.star_proj_fwd(other, types_dev(np.arange(300) % 4), Xo, Wo)
        torch.cuda.synchronize()


# ---- the tensor-power law Q_2^(x)2 (q = 4; the paper's pilot law) ------------------

def _interval_types(M, q=4, period=768):
    """The pilot's interval schedule: type = floor((p mod period) / (period / q))."""
    return ((np.arange(M) % period) // (period // q)).astype(np.int32)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype,out", [("f32", "f32"), ("bf16", "f32"), ("bf16", "bf16")])
@pytest.mark.parametrize("q,s,r,M,types", [
    (4, [192] * 4, [768] * 4, 2048, "interval"),       # the FFN up shape, pipelined kernel
    (4, [768] * 4, [192] * 4, 1100, "random"),         # the FFN down shape
    (4, [72, 40, 96, 64], [136, 200, 56, 96], 777, "random"),
    (4, [32] * 4, [48] * 4, 300, "missing"),           # one type class empty
    (2, [136, 120], [200, 56], 333, "cyclic"),          # L = 1: the two-group law
])
def test_tensor2_fwd_parity(P, dtype, out, q, s, r, M, types):
    import torch
    ga, oa = algs(P, q, s, r, "tensor2")
    seed = 600 + q + M
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, dtype)
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.05, dtype)
    bias = synth.gaussian(seed, 2, (oa.N,), 0.02, "f32")
    if types == "interval":
        t = _interval_types(M, q)
    elif types == "cyclic":
        t = synth.cyclic_types(M, q)
    else:
        t = np.random.default_rng([seed, 3]).integers(0, q, M).astype(np.int32)
        if types == "missing":
            t[t == 1] = 2
    odt = torch.float32 if out == "f32" else torch.bfloat16
    Y, Z = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), f32_dev(bias.exact), "gelu",
                           Z_out=True, out_dtype=odt)
    refY, refZ, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact, bias.exact, "gelu", want_z=True)
    tol = TOL_F32 if (dtype == "f32" and out == "f32") else TOL_BF16
    assert rel_fro(to_host(Z), refZ) <= tol
    assert rel_fro(to_host(Y), refY) <= tol


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("q,s,r,M", [(4, [192] * 4, [768] * 4, 1500), (4, [40, 96, 64, 72], [56, 128, 80, 200], 611)])
def test_tensor2_bwd_data_parity(P, dtype, fused, q, s, r, M):
    import torch
    ga, oa = algs(P, q, s, r, "tensor2")
    seed = 700 + M
    dY = synth.gaussian(seed, 0, (M, oa.N), 1.0, dtype)
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.05, dtype)
    Zp = synth.gaussian(seed, 2, (M, oa.K), 1.0, dtype) if fused else None
    t = np.random.default_rng([seed, 3]).integers(0, q, M).astype(np.int32)
    dX = P.star_proj_bwd_data(ga, types_dev(t), to_dev(dY), to_dev(W),
                              Z_prev=to_dev(Zp) if fused else None,
                              act_prev="gelu" if fused else "none", out_dtype=torch.float32)
    ref = oracle.proj_bwd_data(oa, t, dY.exact, W.exact, Zprev=Zp.exact if fused else None,
                               act_prev="gelu" if fused else "none")
    assert rel_fro(to_host(dX), ref) <= bar(dtype)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("q,s,r,M", [(4, [192] * 4, [768] * 4, 4100), (4, [40, 64, 24, 72], [48, 16, 136, 64], 2049)])
def test_tensor2_bwd_weight_parity(P, dtype, q, s, r, M):
    """Off-diagonal blocks contract over two or four type classes (two ranges
    of type-sorted positions for some blocks), cut into deterministic splits."""
    ga, oa = algs(P, q, s, r, "tensor2")
    seed = 800 + M
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, dtype)
    dY = synth.gaussian(seed, 1, (M, oa.N), 1.0, dtype)
    t = np.random.default_rng([seed, 3]).integers(0, q, M).astype(np.int32)
    dW, db = P.star_proj_bwd_weight(ga, types_dev(t), to_dev(X), to_dev(dY))
    rW, rb = oracle.proj_bwd_weight(oa, t, X.exact, dY.exact)
    assert rel_fro(to_host(dW), rW) <= bar(dtype)
    assert rel_fro(to_host(db), rb) <= bar(dtype)
    dW2, db2 = P.star_proj_bwd_weight(ga, types_dev(t), to_dev(X), to_dev(dY))
    assert np.array_equal(to_host(dW2), to_host(dW)) and np.array_equal(to_host(db2), to_host(db))


@pytest.mark.gpu
def test_tensor2_ffn_train_step_parity(P):
    import torch
    q, D, F, M = 4, 256, 1024, 1000
    up_g, up_o = algs(P, q, [D // q] * q, [F // q] * q, "tensor2")
    dn_g, dn_o = algs(P, q, [F // q] * q, [D // q] * q, "tensor2")
    seed = 900
    X = synth.gaussian(seed, 0, (M, D), 1.0, "bf16")
    Wu = synth.gaussian(seed, 1, (D, F), 0.02, "bf16")
    Wd = synth.gaussian(seed, 2, (F, D), 0.02, "bf16")
    bu = synth.gaussian(seed, 3, (F,), 0.02, "f32")
    bd = synth.gaussian(seed, 4, (D,), 0.02, "f32")
    dY = synth.gaussian(seed, 5, (M, D), 1.0, "bf16")
    t = _interval_types(M, q, 256)
    td = types_dev(t)
    Z, H, Y = P.star_ffn_fwd(up_g, dn_g, td, to_dev(X), to_dev(Wu), f32_dev(bu.exact), to_dev(Wd),
                             f32_dev(bd.exact), "gelu", out_dtype=torch.float32)
    rZ, rH, rY = oracle.ffn_fwd(up_o, dn_o, t, X.exact, Wu.exact, bu.exact, Wd.exact, bd.exact)
    assert rel_fro(to_host(Z), rZ) <= TOL_BF16
    assert rel_fro(to_host(H), rH) <= TOL_BF16
    assert rel_fro(to_host(Y), rY) <= TOL_BF16
    g = P.star_ffn_bwd(up_g, dn_g, td, to_dev(X), Z, H, to_dev(Wu), to_dev(Wd), to_dev(dY), "gelu")
    ref = oracle.ffn_bwd(up_o, dn_o, t, X.exact, rZ, rH, Wu.exact, Wd.exact, dY.exact)
    for k in ("dZ", "dX", "dW_up", "db_up", "dW_down", "db_down"):
        assert rel_fro(to_host(g[k]), ref[k]) <= TOL_BF16, k


@pytest.mark.gpu
@pytest.mark.parametrize("M", [1, 8, 40])
def test_tensor2_decode_parity(P, M):
    import torch
    q, D, F, L = 4, 256, 1024, 3
    up_g, up_o = algs(P, q, [D // q] * q, [F // q] * q, "tensor2")
    dn_g, dn_o = algs(P, q, [F // q] * q, [D // q] * q, "tensor2")
    seed = 950 + M
    Wu = [synth.gaussian(seed, 10 + l, (D, F), 0.02, "bf16") for l in range(L)]
    Wd = [synth.gaussian(seed, 40 + l, (F, D), 0.02, "bf16") for l in range(L)]
    bu = [synth.gaussian(seed, 70 + l, (F,), 0.02, "f32") for l in range(L)]
    bd = [synth.gaussian(seed, 100 + l, (D,), 0.02, "f32") for l in range(L)]
    X = synth.gaussian(seed, 1, (M, D), 1.0, "bf16")
    t = ((synth.decode_positions(seed, M) % 768) // 192).astype(np.int32)
    Y = P.star_decode(up_g, dn_g, types_dev(t), to_dev(X), [to_dev(w) for w in Wu],
                      [f32_dev(b.exact) for b in bu], [to_dev(w) for w in Wd],
                      [f32_dev(b.exact) for b in bd], "gelu", True, out_dtype=torch.float32)
    ref = oracle.decode_stack(up_o, dn_o, t, X.exact, [w.exact for w in Wu], [b.exact for b in bu],
                              [w.exact for w in Wd], [b.exact for b in bd])
    assert rel_fro(to_host(Y), ref) <= TOL_BF16


def test_tensor2_full_size_sampled(P):
    """The bench's tensor-square workload at full size (M = 8192, 768 -> 3072 in
    groups 192 / 768, bias + GELU, interval types), through the planned entry
    point as the bench launches it; sampled rows against the oracle."""
    M, K, N, q = 8192, 768, 3072, 4
    ga, oa = algs(P, q, [192] * 4, [768] * 4, "tensor2")
    X = synth.gaussian(6, 0, (M, K), 1.0, "bf16")
    W = synth.gaussian(6, 1, (K, N), 0.02, "bf16")
    b = synth.gaussian(6, 2, (N,), 0.02, "f32")
    t = _interval_types(M, q)
    plan = P.star_type_plan(q, types_dev(t))
    Y = P.star_proj_fwd_planned(ga, plan, to_dev(X), to_dev(W), f32_dev(b.exact), "gelu")
    rows = _sample_rows(M, 300, 6)
    ref, _, _, _ = oracle.proj_fwd(oa, t[rows], X.exact[rows], W.exact, b.exact, "gelu")
    assert rel_fro(to_host(Y[rows]), ref) <= TOL_BF16


# ---- gated FFN (SwiGLU) -------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_swiglu_elementwise(P, dtype):
    import torch
    n = 4096 * 3
    Zg = synth.gaussian(61, 0, (n,), 2.0, dtype)
    Zu = synth.gaussian(61, 1, (n,), 1.0, dtype)
    dH = synth.gaussian(61, 2, (n,), 1.0, dtype)
    H = P.star_swiglu_fwd(to_dev(Zg), to_dev(Zu))
    ref = oracle.act("silu", Zg.exact) * Zu.exact
    assert rel_fro(to_host(H), ref) <= bar(dtype)
    dZg, dZu = P.star_swiglu_bwd(to_dev(dH), to_dev(Zg), to_dev(Zu))
    assert rel_fro(to_host(dZg), dH.exact * Zu.exact * oracle.act_grad("silu", Zg.exact)) <= bar(dtype)
    assert rel_fro(to_host(dZu), dH.exact * oracle.act("silu", Zg.exact)) <= bar(dtype)
    a = to_dev(Zg)
    out = P.star_add(a, to_dev(Zu), out=a)  # in place
    assert rel_fro(to_host(out), Zg.exact + Zu.exact) <= bar(dtype)


@pytest.mark.parametrize("q,law,bias", [(2, "star", True), (4, "tensor2", False), (2, "dense", True)])
def test_swiglu_ffn_train_step_parity(P, q, law, bias):
    """Gated FFN forward and backward (three projections with one plan, the
    elementwise gate, the summed input gradient) against the oracle."""
    import torch
    D, F, M = 256, 512, 1000
    up_g, up_o = algs(P, q, [D // q] * q, [F // q] * q, law)
    dn_g, dn_o = algs(P, q, [F // q] * q, [D // q] * q, law)
    seed = 970 + q
    X = synth.gaussian(seed, 0, (M, D), 1.0, "bf16")
    Wg = synth.gaussian(seed, 1, (D, F), 0.05, "bf16")
    Wu = synth.gaussian(seed, 2, (D, F), 0.05, "bf16")
    Wd = synth.gaussian(seed, 3, (F, D), 0.05, "bf16")
    bg = synth.gaussian(seed, 4, (F,), 0.02, "f32") if bias else None
    bu = synth.gaussian(seed, 5, (F,), 0.02, "f32") if bias else None
    bd = synth.gaussian(seed, 6, (D,), 0.02, "f32") if bias else None
    dY = synth.gaussian(seed, 7, (M, D), 1.0, "bf16")
    t = _interval_types(M, q, 256) if law == "tensor2" else synth.sequence_types(M, q, 256)
    td = types_dev(t)
    dev_b = lambda b: f32_dev(b.exact) if b is not None else None
    ex_b = lambda b: b.exact if b is not None else None
    Zg, Zu, H, Y = P.star_swiglu_ffn_fwd(up_g, dn_g, td, to_dev(X), to_dev(Wg), dev_b(bg), to_dev(Wu),
                                         dev_b(bu), to_dev(Wd), dev_b(bd), out_dtype=torch.float32)
    rZg, rZu, rH, rY = oracle.swiglu_ffn_fwd(up_o, dn_o, t, X.exact, Wg.exact, ex_b(bg), Wu.exact,
                                             ex_b(bu), Wd.exact, ex_b(bd))
    for got, ref, k in ((Zg, rZg, "Zg"), (Zu, rZu, "Zu"), (H, rH, "H"), (Y, rY, "Y")):
        assert rel_fro(to_host(got), ref) <= TOL_BF16, k
    g = P.star_swiglu_ffn_bwd(up_g, dn_g, td, to_dev(X), Zg, Zu, H, to_dev(Wg), to_dev(Wu), to_dev(Wd),
                              to_dev(dY))
    ref = oracle.swiglu_ffn_bwd(up_o, dn_o, t, X.exact, rZg, rZu, rH, Wg.exact, Wu.exact, Wd.exact, dY.exact)
    for k in ("dZ_gate", "dZ_up", "dX", "dW_gate", "db_gate", "dW_up", "db_up", "dW_down", "db_down"):
        assert rel_fro(to_host(g[k]), ref[k]) <= TOL_BF16, k


@pytest.mark.parametrize("law,q,D,F,L,M", [
    ("star", 2, 256, 1024, 3, 1), ("star", 2, 256, 1024, 3, 8), ("star", 2, 256, 1024, 3, 40),
    ("tensor2", 4, 256, 1024, 3, 1), ("tensor2", 4, 256, 1024, 3, 33), ("dense", 2, 256, 1024, 2, 8),
    ("tensor2", 4, 768, 1536, 12, 1), ("tensor2", 4, 768, 1536, 12, 48),   # the pilot's FFN
])
def test_decode_gated_parity(P, law, q, D, F, L, M):
    import torch
    up_g, up_o = algs(P, q, [D // q] * q, [F // q] * q, law)
    dn_g, dn_o = algs(P, q, [F // q] * q, [D // q] * q, law)
    seed = 990 + M + L
    W = {k: [synth.gaussian(seed, off + l, shp, 0.02, "bf16") for l in range(L)]
         for k, off, shp in (("g", 10, (D, F)), ("u", 40, (D, F)), ("d", 70, (F, D)))}
    b = {k: [synth.gaussian(seed, off + l, (n,), 0.02, "f32") for l in range(L)]
         for k, off, n in (("g", 100, F), ("u", 130, F), ("d", 160, D))}
    X = synth.gaussian(seed, 1, (M, D), 1.0, "bf16")
    pos = synth.decode_positions(seed, M)
    t = (((pos % 768) // 192) if law == "tensor2" else (pos % q)).astype(np.int32)
    dev = lambda k: [to_dev(w) for w in W[k]]
    devb = lambda k: [f32_dev(x.exact) for x in b[k]]
    Y = P.star_decode_gated(up_g, dn_g, types_dev(t), to_dev(X), dev("g"), devb("g"), dev("u"), devb("u"),
                            dev("d"), devb("d"), True, out_dtype=torch.float32)
    ex = lambda k: [w.exact for w in W[k]]
    exb = lambda k: [x.exact for x in b[k]]
    ref = oracle.decode_stack_gated(up_o, dn_o, t, X.exact, ex("g"), exb("g"), ex("u"), exb("u"), ex("d"),
                                    exb("d"))
    assert rel_fro(to_host(Y), ref) <= TOL_BF16
    Y2 = P.star_decode_gated(up_g, dn_g, types_dev(t), to_dev(X), dev("g"), devb("g"), dev("u"), devb("u"),
                             dev("d"), devb("d"), True, out_dtype=torch.float32)
    assert torch.equal(Y, Y2)


def test_decode_gated_refuses_what_does_not_fit(P):
    """Three weight slots do not fit LDS at D = 768 beyond 52 rows: refused
    before any launch, and the plain stack still takes the same shape."""
    import torch
    q, D, F, M = 4, 768, 1536, 64
    up_g, _ = algs(P, q, [D // q] * q, [F // q] * q, "tensor2")
    dn_g, _ = algs(P, q, [F // q] * q, [D // q] * q, "tensor2")
    w = lambda shp: torch.zeros(shp, dtype=torch.bfloat16, device="cuda")
    X = w((M, D))
    t = types_dev(np.zeros(M, np.int32))
    with pytest.raises(RuntimeError, match="unsupported|not supported"):
        P.star_decode_gated(up_g, dn_g, t, X, [w((D, F))], None, [w((D, F))], None, [w((F, D))], None)
    P.star_decode(up_g, dn_g, t, X, [w((D, F))], None, [w((F, D))], None, "gelu")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_max_q_narrow_groups(P, dtype):
    """q = 64 (the largest the ABI takes) with 8-wide groups: every tile spans
    many groups' worth of classes; forward, activation and weight gradients."""
    import torch
    q, w, M = 64, 8, 1000
    ga, oa = algs(P, q, [w] * q, [w] * q)
    X = synth.gaussian(77, 0, (M, q * w), 1.0, dtype)
    W = synth.gaussian(77, 1, (q * w, q * w), 0.1, dtype)
    dY = synth.gaussian(77, 2, (M, q * w), 1.0, dtype)
    t = np.random.default_rng([77, 3]).integers(0, q, M).astype(np.int32)
    Y = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), out_dtype=torch.float32)
    ref, _, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact)
    assert rel_fro(to_host(Y), ref) <= bar(dtype)
    dX = P.star_proj_bwd_data(ga, types_dev(t), to_dev(dY), to_dev(W), out_dtype=torch.float32)
    assert rel_fro(to_host(dX), oracle.proj_bwd_data(oa, t, dY.exact, W.exact)) <= bar(dtype)
    dW, db = P.star_proj_bwd_weight(ga, types_dev(t), to_dev(X), to_dev(dY))
    rW, rb = oracle.proj_bwd_weight(oa, t, X.exact, dY.exact)
    assert rel_fro(to_host(dW), rW) <= bar(dtype)
    assert rel_fro(to_host(db), rb) <= bar(dtype)


@pytest.mark.parametrize("case", ["many_layers", "other_groups"])
def test_decode_per_projection_path(P, case):
    """Shapes the persistent stack does not take run one launch per projection:
    more layers than the stack holds (33), or a down projection whose output
    groups differ from the up projection's input groups."""
    import torch
    if case == "many_layers":
        q, L, M = 2, 33, 5
        up_g, up_o = algs(P, q, [64, 64], [128, 128])
        dn_g, dn_o = algs(P, q, [128, 128], [64, 64])
    else:
        q, L, M = 2, 3, 9
        up_g, up_o = algs(P, q, [64, 64], [128, 128])
        dn_g, dn_o = algs(P, q, [128, 128], [40, 88])
    D, F = up_o.K, up_o.N
    seed = 1100 + L
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


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tanh_gelu_paths(P, dtype):
    """The tanh form of GELU in the forward epilogue, in the activation
    gradient's fused derivative and in the decode stack."""
    import torch
    q = 2
    ga, oa = algs(P, q, [192, 192], [384, 384])
    M = 700
    seed = 1200
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, dtype)
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.05, dtype)
    b = synth.gaussian(seed, 2, (oa.N,), 0.02, "f32")
    t = np.random.default_rng([seed, 3]).integers(0, q, M).astype(np.int32)
    Y = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), f32_dev(b.exact), "gelu_tanh",
                        out_dtype=torch.float32)
    ref, _, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact, b.exact, "gelu_tanh")
    assert rel_fro(to_host(Y), ref) <= bar(dtype)
    dY = synth.gaussian(seed, 4, (M, oa.N), 1.0, dtype)
    Zp = synth.gaussian(seed, 5, (M, oa.K), 1.0, dtype)
    dX = P.star_proj_bwd_data(ga, types_dev(t), to_dev(dY), to_dev(W), Z_prev=to_dev(Zp),
                              act_prev="gelu_tanh", out_dtype=torch.float32)
    refd = oracle.proj_bwd_data(oa, t, dY.exact, W.exact, Zprev=Zp.exact, act_prev="gelu_tanh")
    assert rel_fro(to_host(dX), refd) <= bar(dtype)
    if dtype == "bf16":
        up_g, up_o = algs(P, q, [64, 64], [256, 256])
        dn_g, dn_o = algs(P, q, [256, 256], [64, 64])
        L, Md = 2, 3
        Wu = [synth.gaussian(seed, 10 + l, (128, 512), 0.05, "bf16") for l in range(L)]
        Wd = [synth.gaussian(seed, 20 + l, (512, 128), 0.05, "bf16") for l in range(L)]
        Xd = synth.gaussian(seed, 30, (Md, 128), 1.0, "bf16")
        td = np.array([0, 1, 1], np.int32)
        Yd = P.star_decode(up_g, dn_g, types_dev(td), to_dev(Xd), [to_dev(w) for w in Wu], None,
                           [to_dev(w) for w in Wd], None, "gelu_tanh", True, out_dtype=torch.float32)
        refdd = oracle.decode_stack(up_o, dn_o, td, Xd.exact, [w.exact for w in Wu], [None] * L,
                                    [w.exact for w in Wd], [None] * L, act="gelu_tanh")
        assert rel_fro(to_host(Yd), refdd) <= TOL_BF16
