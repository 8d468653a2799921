"""GPU parity of the merged gate/up SwiGLU (§"Kernel Benchmark Details": the
gated comparison merges gate and up; Tab. kernel-ffn) against the fp64
oracle: the merged product X *_q W_gu with SwiGLU in its epilogue, the
elementwise SwiGLU on a merged output, and the complete gated FFN built from
them.

The oracle side is the plain definition: the gate and up projections as two
separate products (``oracle.proj_fwd`` of the up layout with W_gate and
W_up), H = silu(Z_g) . Z_u; only the GPU side sees the interleaved layout,
so a wrong interleave, a swapped gate and up, or a dropped bias shows up.
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


def _interleave(g, u):
    """Reference interleave of the last axis in 8-wide chunks (numpy)."""
    lead, F = g.shape[:-1], g.shape[-1]
    out = np.empty(lead + (2 * F,), dtype=g.dtype)
    for c in range(F // 8):
        out[..., 16 * c:16 * c + 8] = g[..., 8 * c:8 * c + 8]
        out[..., 16 * c + 8:16 * c + 16] = u[..., 8 * c:8 * c + 8]
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_swiglu_merged_elementwise(P, dtype):
    M, F = 37, 8 * 53
    Z = synth.gaussian(71, 0, (M, 2 * F), 2.0, dtype)
    H = P.star_swiglu_merged_fwd(to_dev(Z))
    g = np.concatenate([Z.exact[:, 16 * c:16 * c + 8] for c in range(F // 8)], axis=1)
    u = np.concatenate([Z.exact[:, 16 * c + 8:16 * c + 16] for c in range(F // 8)], axis=1)
    ref = oracle.act("silu", g) * u
    assert rel_fro(to_host(H), ref) <= (TOL_F32 if dtype == "f32" else TOL_BF16)


def _types(kind, M, q, seed):
    rng = np.random.default_rng([seed, 9])
    if kind == "cyclic":
        return synth.cyclic_types(M, q)
    t = rng.integers(0, q, M).astype(np.int32)
    if kind == "gaps":
        t[t == 1] = 0
        t[M // 2] = 1 if q > 2 else t[M // 2]
    return t


# (law, q, s, r (the up layout's output widths), M, types)
CASES = [
    ("star", 32, [64] * 32, [96] * 32, 1500, "random"),    # merged 192: a full and a half tile
    ("star", 4, [136, 64, 200, 72], [128, 64, 32, 96], 700, "gaps"),
    ("star", 32, [64] * 32, [24] * 32, 1000, "random"),    # merged 48: part of one tile
    ("dense", 8, [64] * 8, [64] * 8, 300, "random"),
    ("tensor2", 4, [72, 64, 136, 64], [104, 64, 128, 40], 500, "random"),
    ("star", 128, [16] * 128, [32] * 128, 2000, "random"),  # q above 64
]


@pytest.mark.parametrize("out", ["f32", "bf16"])
@pytest.mark.parametrize("law,q,s,r,M,types", CASES)
def test_swiglu_up_fused_parity(P, out, law, q, s, r, M, types):
    import torch
    up = oracle.Alg(q, tuple(s), tuple(r), law)
    ga = P.Algebra(q, s, r, law).merged_gate_up()
    seed = 3100 + q + M
    X = synth.gaussian(seed, 0, (M, up.K), 1.0, "bf16")
    Wg = synth.gaussian(seed, 1, (up.K, up.N), 0.05, "bf16")
    Wu = synth.gaussian(seed, 2, (up.K, up.N), 0.05, "bf16")
    bg = synth.gaussian(seed, 3, (up.N,), 0.1, "f32")
    bu = synth.gaussian(seed, 4, (up.N,), 0.1, "f32")
    t = _types(types, M, q, seed)
    Zg, _, _, _ = oracle.proj_fwd(up, t, X.exact, Wg.exact, bg.exact)
    Zu, _, _, _ = oracle.proj_fwd(up, t, X.exact, Wu.exact, bu.exact)
    Href = oracle.act("silu", Zg) * Zu
    W_gu = P.pack_gate_up(to_dev(Wg), to_dev(Wu))
    b_gu = P.pack_gate_up(f32_dev(bg.exact), f32_dev(bu.exact))
    plan = P.star_type_plan(q, types_dev(t))
    odt = torch.float32 if out == "f32" else torch.bfloat16
    H, Z = P.star_swiglu_up_fwd_planned(ga, plan, to_dev(X), W_gu, b_gu, Z_out=True, out_dtype=odt)
    assert rel_fro(to_host(Z), _interleave(Zg, Zu)) <= TOL_BF16
    gH = to_host(H)
    assert rel_fro(gH, Href) <= TOL_BF16
    live = np.linalg.norm(Href, axis=1) > 0
    diff = np.linalg.norm(gH - Href, axis=1)[live] / np.linalg.norm(Href, axis=1)[live]
    assert diff.max() <= 4 * TOL_BF16
    # without the pre-activation and without a bias
    H2 = P.star_swiglu_up_fwd_planned(ga, plan, to_dev(X), W_gu, out_dtype=odt)
    Zg0, _, _, _ = oracle.proj_fwd(up, t, X.exact, Wg.exact)
    Zu0, _, _, _ = oracle.proj_fwd(up, t, X.exact, Wu.exact)
    assert rel_fro(to_host(H2), oracle.act("silu", Zg0) * Zu0) <= TOL_BF16


@pytest.mark.parametrize("q", [4, 32])
def test_gated_ffn_merged_matches_oracle(P, q):
    """The complete gated FFN: fused merged gate/up, then the down product.
    The oracle mirrors what the GPU path stores in bf16: H (the down
    product's input) is rounded, the pre-activations are not (the fused
    epilogue applies SwiGLU to the fp32 accumulators)."""
    D, F, M = 64 * q, 96 * q, 1024
    up, down = oracle.Alg.equal(q, D, F), oracle.Alg.equal(q, F, D)
    ga_up, ga_dn = P.Algebra.equal(q, D, F), P.Algebra.equal(q, F, D)
    seed = 3200 + q
    X = synth.gaussian(seed, 0, (M, D), 1.0, "bf16")
    Wg = synth.gaussian(seed, 1, (D, F), 0.05, "bf16")
    Wu = synth.gaussian(seed, 2, (D, F), 0.05, "bf16")
    Wd = synth.gaussian(seed, 3, (F, D), 0.05, "bf16")
    t = synth.cyclic_types(M, q)
    Zg, _, _, _ = oracle.proj_fwd(up, t, X.exact, Wg.exact)
    Zu, _, _, _ = oracle.proj_fwd(up, t, X.exact, Wu.exact)
    Yref, _, _, _ = oracle.proj_fwd(down, t, oracle.round_bf16(oracle.act("silu", Zg) * Zu), Wd.exact)
    plan = P.star_type_plan(q, types_dev(t))
    H = P.star_swiglu_up_fwd_planned(ga_up.merged_gate_up(), plan, to_dev(X), P.pack_gate_up(to_dev(Wg), to_dev(Wu)))
    Y = P.star_proj_fwd_planned(ga_dn, plan, H, to_dev(Wd))
    assert rel_fro(to_host(Y), Yref) <= TOL_BF16


def _sample_rows(M, n, seed):
    rng = np.random.default_rng([seed, 11])
    return np.unique(np.concatenate([[0, 1, M - 2, M - 1], rng.choice(M, n, replace=False)]))


# The SwiGLU comparison's shapes at full size (Tab. kernel-ffn, q = 32,
# M = 2048): the fused merged gate/up and the down product over all rows,
# checked against the oracle on sampled rows (every step is row-local).
@pytest.mark.parametrize("name,D,F", [("Qwen3-8B", 4096, 12288), ("DeepSeek-V3 expert", 7168, 2048)])
def test_gated_ffn_merged_kernel_study_sampled(P, name, D, F):
    import torch
    q, M = 32, 2048
    up, down = oracle.Alg.equal(q, D, F), oracle.Alg.equal(q, F, D)
    ga_up, ga_dn = P.Algebra.equal(q, D, F), P.Algebra.equal(q, F, D)
    seed = 3300 + D
    X = synth.gaussian(seed, 0, (M, D), 1.0, "bf16")
    Wg = synth.gaussian(seed, 1, (D, F), (1.0 / D) ** 0.5, "bf16")
    Wu = synth.gaussian(seed, 2, (D, F), (1.0 / D) ** 0.5, "bf16")
    Wd = synth.gaussian(seed, 3, (F, D), (1.0 / F) ** 0.5, "bf16")
    t = synth.cyclic_types(M, q)
    plan = P.star_type_plan(q, types_dev(t))
    H = P.star_swiglu_up_fwd_planned(ga_up.merged_gate_up(), plan, to_dev(X), P.pack_gate_up(to_dev(Wg), to_dev(Wu)))
    Y = P.star_proj_fwd_planned(ga_dn, plan, H, to_dev(Wd))
    rows = _sample_rows(M, 160, seed)
    got = to_host(Y[rows])
    del H, Y
    torch.cuda.empty_cache()
    Zg, _, _, _ = oracle.proj_fwd(up, t[rows], X.exact[rows], Wg.exact)
    Zu, _, _, _ = oracle.proj_fwd(up, t[rows], X.exact[rows], Wu.exact)
    Yref, _, _, _ = oracle.proj_fwd(down, t[rows], oracle.round_bf16(oracle.act("silu", Zg) * Zu), Wd.exact)
    assert rel_fro(got, Yref) <= TOL_BF16
