"""GPU parity of the forward product with many small groups (Sec. "Kernel
Scaling on Transformer Shapes"): the tiles of 64 rows x 128 columns that
carry q up to 256 at the widths of the paper's projection study, against the
fp64 oracle on the same seeded inputs.

Each case runs the same inputs through every tile size (forced with
star_set_fwd_tiles: 64 x 128, 256 x 256 and 256 x 192) and through the
automatic choice, and covers: several
tiles per workgroup (the copy stream runs across tile boundaries), one-step
tiles (groups 64 wide; under the graph law a diagonal-only tile contracts a
single group and the tiles of non-edges are skipped), K tails (input widths
not multiples of 64), column tails (output widths not multiples of 128),
empty and one-row types, every law, bias, GELU and the pre-activation, fp32
and bf16 outputs, q = 128 and 256 (K steps spanning several 8- to 40-wide
groups), and the paper's projection shapes at full size on sampled rows (the
product is row-local).
"""

import numpy as np
import pytest

import oracle
import synth
from helpers import TOL_BF16, f32_dev, rel_fro, to_dev, to_host, types_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    assert torch.cuda.is_available(), "GPU parity tests need a GPU"
    import paper_2609_32814_amd as P
    yield P
    P.star_set_fwd_tiles("auto")


def _types(kind, M, q, seed):
    rng = np.random.default_rng([seed, 7])
    if kind == "cyclic":
        return synth.cyclic_types(M, q)
    t = rng.integers(0, q, M).astype(np.int32)
    if kind == "gaps":  # two empty types and a one-row type
        t[t == 1] = 0
        t[t == q - 2] = q - 1
        t[t == 3] = 2
        t[M // 3] = 3
    return t


def _run_all_tiles(P, ga, t, X, W, b, act, want_z, odt):
    out = {}
    for tiles in ("small", "wide", "wide192", "auto"):
        P.star_set_fwd_tiles(tiles)
        try:
            res = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), None if b is None else f32_dev(b.exact),
                                  act, Z_out=want_z, out_dtype=odt)
        finally:
            P.star_set_fwd_tiles("auto")
        out[tiles] = res if want_z else (res, None)
    return out


def _s(widths, q):
    return [widths[g % len(widths)] for g in range(q)]


# (law, q, s, r, M, types)
CASES = [
    # 48 column tiles x 32 row blocks: three tiles per workgroup
    ("star", 16, [128] * 16, [384] * 16, 2048, "cyclic"),
    # 64-wide groups: two one-step products per tile; 47 rows a type
    ("star", 32, [64] * 32, [64] * 32, 1500, "random"),
    # K tails of 8..56 past a multiple of 64, column tails, empty types
    ("star", 24, _s([72, 136, 200, 64, 8 * 13], 24), _s([136, 8, 264, 128, 72], 24), 900, "gaps"),
    ("dense", 12, _s([72, 64, 136], 12), _s([200, 64, 136, 8], 12), 700, "gaps"),
    ("tensor2", 4, [136, 64, 200, 72], [264, 128, 72, 136], 300, "random"),
    # the largest q: half-empty 64-row tiles, 8 tiles per workgroup
    ("star", 64, [64] * 64, [128] * 64, 2048, "cyclic"),
]


@pytest.mark.parametrize("out", ["f32", "bf16"])
@pytest.mark.parametrize("law,q,s,r,M,types", CASES)
def test_small_tiles_bias_gelu(P, out, law, q, s, r, M, types):
    import torch
    ga, oa = P.Algebra(q, s, r, law), oracle.Alg(q, tuple(s), tuple(r), law)
    seed = 2100 + q + M
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, "bf16")
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.03, "bf16")
    b = synth.gaussian(seed, 2, (oa.N,), 0.05, "f32")
    t = _types(types, M, q, seed)
    odt = torch.float32 if out == "f32" else torch.bfloat16
    refY, refZ, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact, b.exact, "gelu", want_z=True)
    for tiles, (Y, Z) in _run_all_tiles(P, ga, t, X, W, b, "gelu", True, odt).items():
        gY, gZ = to_host(Y), to_host(Z)
        assert rel_fro(gZ, refZ) <= TOL_BF16, tiles
        assert rel_fro(gY, refY) <= TOL_BF16, tiles
        # row by row: a dropped, repeated or misplaced tile shows up here
        live = np.linalg.norm(refZ, axis=1) > 0
        diff = np.linalg.norm(gZ - refZ, axis=1)[live] / np.linalg.norm(refZ, axis=1)[live]
        assert diff.max() <= 4 * TOL_BF16, tiles


def test_small_tiles_without_bias(P):
    q, M = 32, 777
    ga, oa = P.Algebra.equal(q, 128 * q, 192 * q), oracle.Alg.equal(q, 128 * q, 192 * q)
    X = synth.gaussian(2200, 0, (M, oa.K), 1.0, "bf16")
    W = synth.gaussian(2200, 1, (oa.K, oa.N), 0.03, "bf16")
    t = _types("random", M, q, 2200)
    ref, _, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact)
    for tiles, (Y, _) in _run_all_tiles(P, ga, t, X, W, None, "none", False, None).items():
        assert rel_fro(to_host(Y), ref) <= TOL_BF16, tiles


@pytest.mark.parametrize("M", [1, 31, 65])
def test_small_tiles_few_rows(P, M):
    q = 32
    ga, oa = P.Algebra.equal(q, 64 * q, 136 * q), oracle.Alg.equal(q, 64 * q, 136 * q)
    X = synth.gaussian(2300 + M, 0, (M, oa.K), 1.0, "bf16")
    W = synth.gaussian(2300 + M, 1, (oa.K, oa.N), 0.03, "bf16")
    b = synth.gaussian(2300 + M, 2, (oa.N,), 0.05, "f32")
    t = _types("random", M, q, 2300 + M)
    ref, _, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact, b.exact, "gelu")
    for tiles, (Y, _) in _run_all_tiles(P, ga, t, X, W, b, "gelu", False, None).items():
        assert rel_fro(to_host(Y), ref) <= TOL_BF16, tiles


def test_small_tiles_graph_law(P):
    """q = 16, groups 64 wide: a type's tile of its own group contracts one
    group (one K step), an edge tile two, a non-edge tile none (skipped; the
    fill kernel writes act(bias) there)."""
    import torch
    q, M = 16, 2000
    E = (np.random.default_rng([2400, q]).random((q, q)) < 0.3).astype(np.uint8)
    np.fill_diagonal(E, 0)
    s, r = [64] * q, _s([64, 192, 136], q)
    ga = P.Algebra(q, s, r, "graph", E)
    oa = oracle.Alg(q, tuple(s), tuple(r), "graph", tuple(map(tuple, E)))
    X = synth.gaussian(2400, 0, (M, oa.K), 1.0, "bf16")
    W = synth.gaussian(2400, 1, (oa.K, oa.N), 0.03, "bf16")
    b = synth.gaussian(2400, 2, (oa.N,), 0.05, "f32")
    t = _types("random", M, q, 2400)
    refY, refZ, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact, b.exact, "gelu", want_z=True)
    for tiles, (Y, Z) in _run_all_tiles(P, ga, t, X, W, b, "gelu", True, torch.float32).items():
        assert rel_fro(to_host(Z), refZ) <= TOL_BF16, tiles
        assert rel_fro(to_host(Y), refY) <= TOL_BF16, tiles


# q above 64 (the star and dense laws): groups 8 to 40 wide, so a 64-deep K
# step spans both ranges of a tile's contraction or several groups
LARGE_Q = [
    ("star", 128, [16] * 128, [40] * 128, 3000, "random"),
    ("star", 256, _s([8, 16, 24, 40], 256), _s([8, 24, 136, 96], 256), 2000, "gaps"),
    ("dense", 128, [16] * 128, [8] * 128, 400, "random"),
]


@pytest.mark.parametrize("out", ["f32", "bf16"])
@pytest.mark.parametrize("law,q,s,r,M,types", LARGE_Q)
def test_large_q_bias_gelu(P, out, law, q, s, r, M, types):
    import torch
    ga, oa = P.Algebra(q, s, r, law), oracle.Alg(q, tuple(s), tuple(r), law)
    seed = 2600 + q + M
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, "bf16")
    W = synth.gaussian(seed, 1, (oa.K, oa.N), 0.05, "bf16")
    b = synth.gaussian(seed, 2, (oa.N,), 0.05, "f32")
    t = _types(types, M, q, seed)
    odt = torch.float32 if out == "f32" else torch.bfloat16
    refY, refZ, _, _ = oracle.proj_fwd(oa, t, X.exact, W.exact, b.exact, "gelu", want_z=True)
    Y, Z = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W), f32_dev(b.exact), "gelu", Z_out=True,
                           out_dtype=odt)
    gY, gZ = to_host(Y), to_host(Z)
    assert rel_fro(gZ, refZ) <= TOL_BF16
    assert rel_fro(gY, refY) <= TOL_BF16
    live = np.linalg.norm(refZ, axis=1) > 0
    diff = np.linalg.norm(gZ - refZ, axis=1)[live] / np.linalg.norm(refZ, axis=1)[live]
    assert diff.max() <= 4 * TOL_BF16


def test_large_q_refused_where_not_built(P):
    """fp32 operands at q > 64 are refused before anything runs."""
    import torch
    ga = P.Algebra.equal(128, 16 * 128, 16 * 128)
    X = torch.zeros((4, 16 * 128), device="cuda")
    W = torch.zeros((16 * 128, 16 * 128), device="cuda")
    with pytest.raises(Exception, match="UNSUPPORTED|unsupported"):
        P.star_proj_fwd(ga, types_dev(np.zeros(4, np.int32)), X, W)


def _sample_rows(M, n, seed):
    rng = np.random.default_rng([seed, 11])
    return np.unique(np.concatenate([[0, 1, M - 2, M - 1], rng.choice(M, n, replace=False)]))


# The paper's pure expansion projections at M = 2048 (Tab. kernel-products),
# at the q the automatic choice runs on the small tiles.
SHAPES = [
    ("Qwen3-1.7B", 2048, 6144, 32),
    ("Qwen3-8B", 4096, 12288, 32),
    ("Qwen3-30B-A3B expert", 2048, 768, 16),
    ("DeepSeek-V3 expert", 7168, 2048, 16),
]


@pytest.mark.parametrize("name,D,F,q", SHAPES + [("Qwen3-1.7B", 2048, 6144, 128), ("Qwen3-8B", 4096, 12288, 256)])
def test_projection_shapes_full_size_sampled(P, name, D, F, q):
    import torch
    M = 2048
    ga, oa = P.Algebra.equal(q, D, F), oracle.Alg.equal(q, D, F)
    seed = 2500 + q + D
    X = synth.gaussian(seed, 0, (M, D), 1.0, "bf16")
    W = synth.gaussian(seed, 1, (D, F), (1.0 / D) ** 0.5, "bf16")
    t = synth.cyclic_types(M, q)
    Y = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W))
    rows = _sample_rows(M, 160, seed)
    ref, _, _, _ = oracle.proj_fwd(oa, t[rows], X.exact[rows], W.exact)
    assert rel_fro(to_host(Y[rows]), ref) <= TOL_BF16
    del Y
    torch.cuda.empty_cache()


# The kernel study's largest runs (Tab. kernel-products): Qwen3-32B's
# expansion 5120 -> 25600 at M = 8192, q = 128 (groups 40 / 200 wide) and at
# M = 32768, q = 256, where the equal widths 20 / 100 are not multiples of 8
# and alternate 16 / 24 and 96 / 104 (same totals, same block products).
@pytest.mark.parametrize("M,q,s,r", [
    (8192, 128, [40] * 128, [200] * 128),
    (32768, 256, [16, 24] * 128, [96, 104] * 128),
])
def test_qwen3_32b_large_q_full_size_sampled(P, M, q, s, r):
    import torch
    ga, oa = P.Algebra(q, s, r), oracle.Alg(q, tuple(s), tuple(r))
    seed = 2700 + q
    X = synth.gaussian(seed, 0, (M, oa.K), 1.0, "bf16")
    W = synth.gaussian(seed, 1, (oa.K, oa.N), (1.0 / oa.K) ** 0.5, "bf16")
    t = synth.cyclic_types(M, q)
    Y = P.star_proj_fwd(ga, types_dev(t), to_dev(X), to_dev(W))
    rows = _sample_rows(M, 160, seed)
    ref, _, _, _ = oracle.proj_fwd(oa, t[rows], X.exact[rows], W.exact)
    got = to_host(Y[rows])
    del Y
    torch.cuda.empty_cache()
    assert rel_fro(got, ref) <= TOL_BF16
    # every sampled row on its own (each row type reaches 2q - 1 of the q^2 blocks)
    live = np.linalg.norm(ref, axis=1) > 0
    diff = np.linalg.norm(got - ref, axis=1)[live] / np.linalg.norm(ref, axis=1)[live]
    assert diff.max() <= 4 * TOL_BF16
