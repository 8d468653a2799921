"""GPU parity for algebraic attention (appendix "Attention Extension and
Detailed Cost Accounting"): the causal forward (Alg. attention-training, its
score and aggregation steps) and one decode step over a KV cache (Alg.
attention-decoding) through the C ABI, against the fp64 oracle on the same
seeded bf16 inputs.

The shapes span several 128-query blocks and 32-key blocks with ragged
tails, both head widths (64, 128), group widths m from 8 to 128, the star,
dense and tensor-square laws, grouped-query heads (including more than 8
query heads per key/value head, which splits the decode workgroups), and
cyclic, interval and random type schedules.  Edge cases: one position, types
with no positions, positions whose type is out of range, cache lengths of 0,
1, the capacity and beyond it.  The full-size cases sample (sequence, head)
pairs of the 110M-class shapes (16 x 1536 positions, 12 heads of 64) and
check every decode row of 64 sequences at random positions below 2048.

Bar: relative Frobenius error <= 2e-3 against the oracle (bf16 operands,
fp32 softmax and accumulation; the probabilities enter the value product in
bf16), fp32 outputs.  A bf16 output is checked to be exactly the rounding of
the fp32 one.
"""

import numpy as np
import pytest

import oracle
import synth
from helpers import TOL_BF16, rel_fro, to_dev, to_host, types_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    assert torch.cuda.is_available(), "GPU parity tests need a GPU"
    import paper_2609_32814_amd as P
    return P


def schedule(kind, S, q, seed=0):
    p = np.arange(S)
    if kind == "cyclic":
        return (p % q).astype(np.int32)
    if kind == "interval":  # the pilot's schedule: floor((p mod 768) / (768 / q))
        return ((p % 768) // (768 // q)).astype(np.int32)
    if kind == "random":
        return np.random.default_rng([70, S, q, seed]).integers(0, q, S).astype(np.int32)
    raise ValueError(kind)


def inputs(seed, B, S, H, Hkv, D):
    Q = synth.gaussian(seed, 0, (B * S, H * D), 1.0, "bf16")
    K = synth.gaussian(seed, 1, (B * S, Hkv * D), 1.0, "bf16")
    V = synth.gaussian(seed, 2, (B * S, Hkv * D), 1.0, "bf16")
    return Q, K, V


def gpu_fwd(P, shape, pt, Q, K, V, out_dtype=None, want_lse=False, O=None):
    import torch
    B, S, H, Hkv, D = shape.batch, shape.seq_len, shape.n_heads, shape.n_kv_heads, shape.head_dim
    plan = P.star_type_plan(shape.q, types_dev(pt))
    return P.star_attn_fwd(shape, plan, to_dev(Q).view(B, S, H, D), to_dev(K).view(B, S, Hkv, D),
                           to_dev(V).view(B, S, Hkv, D), O=O, out_dtype=out_dtype or torch.float32,
                           want_lse=want_lse)


# (law, q, head_dim, B, S, n_heads, n_kv, schedule)
FWD_CASES = [
    ("star", 2, 64, 2, 300, 4, 2, "cyclic"),
    ("star", 4, 64, 2, 257, 3, 3, "cyclic"),
    ("tensor2", 4, 64, 1, 515, 2, 1, "interval"),
    ("dense", 4, 64, 2, 200, 2, 2, "cyclic"),
    ("star", 8, 64, 1, 190, 2, 2, "random"),      # m = 8: lanes zero their own slice
    ("star", 1, 64, 1, 100, 1, 1, "cyclic"),      # q = 1: ordinary attention
    ("star", 2, 128, 2, 333, 4, 1, "cyclic"),
    ("tensor2", 4, 128, 1, 400, 2, 2, "random"),
    ("star", 16, 128, 1, 160, 2, 2, "cyclic"),    # q = 16, m = 8
    ("star", 4, 64, 1, 1, 2, 2, "cyclic"),        # one position
    ("star", 4, 64, 2, 2, 1, 1, "cyclic"),        # types 2 and 3 have no positions
    ("star", 2, 64, 3, 1025, 2, 2, "random"),     # a ragged tail past 1024
]


def _ids(c):
    return f"{c[0]}-q{c[1]}-d{c[2]}-B{c[3]}-S{c[4]}-h{c[5]}/{c[6]}-{c[7]}"


@pytest.mark.parametrize("case", FWD_CASES, ids=_ids)
def test_attn_fwd_parity(P, case):
    law, q, D, B, S, H, Hkv, kind = case
    m = D // q
    seed = 3000 + S + 7 * q
    Q, K, V = inputs(seed, B, S, H, Hkv, D)
    pt = schedule(kind, S, q, seed)
    shape = P.AttnShape(B, S, H, Hkv, D, q, law)
    O, lse = gpu_fwd(P, shape, pt, Q, K, V, want_lse=True)
    ref, ref_lse = oracle.attn_fwd(q, law, m, H, Hkv, B, S, pt, Q.exact, K.exact, V.exact, want_lse=True)
    got = to_host(O).reshape(B * S, H * D)
    assert rel_fro(got, ref) <= TOL_BF16
    np.testing.assert_allclose(to_host(lse), ref_lse, rtol=0, atol=1e-4)


def test_attn_fwd_bf16_output_is_rounded_fp32(P):
    import torch
    B, S, H, Hkv, D, q = 2, 211, 2, 1, 64, 2
    Q, K, V = inputs(3100, B, S, H, Hkv, D)
    pt = schedule("cyclic", S, q)
    shape = P.AttnShape(B, S, H, Hkv, D, q)
    O32 = gpu_fwd(P, shape, pt, Q, K, V, out_dtype=torch.float32)
    O16 = gpu_fwd(P, shape, pt, Q, K, V, out_dtype=torch.bfloat16)
    assert torch.equal(O16, O32.to(torch.bfloat16))


def test_attn_fwd_deterministic(P):
    import torch
    B, S, H, Hkv, D, q = 2, 390, 3, 3, 128, 4
    Q, K, V = inputs(3200, B, S, H, Hkv, D)
    pt = schedule("random", S, q)
    shape = P.AttnShape(B, S, H, Hkv, D, q, "tensor2")
    a = gpu_fwd(P, shape, pt, Q, K, V)
    b = gpu_fwd(P, shape, pt, Q, K, V)
    assert torch.equal(a, b)


def test_attn_fwd_out_of_range_types(P):
    """A position whose type is outside [0, q) is neither a query nor a key:
    its output rows stay untouched, and every other row equals the oracle on
    the sequence with those positions removed."""
    import torch
    B, S, H, Hkv, D, q = 2, 260, 2, 2, 64, 4
    Q, K, V = inputs(3300, B, S, H, Hkv, D)
    pt = schedule("cyclic", S, q)
    bad = np.zeros(S, bool)
    bad[[0, 5, 77, 128, 129, 259]] = True
    pt_bad = pt.copy()
    pt_bad[bad] = np.array([4, -1, 7, 100, -5, 4])
    shape = P.AttnShape(B, S, H, Hkv, D, q)
    O = torch.full((B, S, H, D), 123.0, dtype=torch.float32, device="cuda")
    gpu_fwd(P, shape, pt_bad, Q, K, V, O=O)
    got = to_host(O)
    assert np.all(got[:, bad] == 123.0)
    keep = ~bad
    Sk = int(keep.sum())
    sel = np.concatenate([b * S + np.nonzero(keep)[0] for b in range(B)])
    ref = oracle.attn_fwd(q, "star", D // q, H, Hkv, B, Sk, pt[keep], Q.exact[sel], K.exact[sel], V.exact[sel])
    assert rel_fro(got[:, keep].reshape(B * Sk, H * D), ref) <= TOL_BF16


@pytest.mark.parametrize("law,kind", [("star", "cyclic"), ("tensor2", "interval"), ("dense", "cyclic")])
def test_attn_fwd_full_size_sampled(P, law, kind):
    """16 sequences x 1536 positions, 12 heads of 64, q = 4: every output is
    computed, sampled (sequence, head) pairs are checked against the oracle
    run on that slice alone."""
    B, S, H, Hkv, D, q = 16, 1536, 12, 12, 64, 4
    m = D // q
    Q, K, V = inputs(3400, B, S, H, Hkv, D)
    pt = schedule(kind, S, q)
    shape = P.AttnShape(B, S, H, Hkv, D, q, law)
    O, lse = gpu_fwd(P, shape, pt, Q, K, V, want_lse=True)
    got = to_host(O)
    gl = to_host(lse)
    Qe, Ke, Ve = (x.exact.reshape(B, S, -1, D) for x in (Q, K, V))
    for b, h in [(0, 0), (15, 11), (7, 5)]:
        ref, rl = oracle.attn_fwd(q, law, m, 1, 1, 1, S, pt, Qe[b, :, h], Ke[b, :, h], Ve[b, :, h], want_lse=True)
        assert rel_fro(got[b, :, h], ref) <= TOL_BF16, (b, h)
        np.testing.assert_allclose(gl[b, h], rl[0, 0], rtol=0, atol=1e-4)
    assert np.all(np.isfinite(got))


# ---- decode ---------------------------------------------------------------------

def gpu_decode(P, shape, pt, L, Qd, Kc, Vc, out_dtype=None):
    import torch
    B, S, H, Hkv, D = shape.batch, shape.seq_len, shape.n_heads, shape.n_kv_heads, shape.head_dim
    return P.star_attn_decode(shape, types_dev(pt), types_dev(L), to_dev(Qd).view(B, H, D),
                              to_dev(Kc).view(B, S, Hkv, D), to_dev(Vc).view(B, S, Hkv, D),
                              out_dtype=out_dtype or torch.float32)


def dec_inputs(seed, B, S, H, Hkv, D):
    Qd = synth.gaussian(seed, 0, (B, H * D), 1.0, "bf16")
    Kc = synth.gaussian(seed, 1, (B, S, Hkv * D), 1.0, "bf16")
    Vc = synth.gaussian(seed, 2, (B, S, Hkv * D), 1.0, "bf16")
    return Qd, Kc, Vc


# (law, q, head_dim, B, S_max, n_heads, n_kv, schedule)
DEC_CASES = [
    ("star", 2, 64, 5, 300, 4, 4, "cyclic"),
    ("star", 4, 64, 3, 700, 12, 12, "cyclic"),
    ("tensor2", 4, 64, 4, 260, 8, 2, "interval"),
    ("star", 2, 128, 3, 200, 4, 1, "cyclic"),
    ("star", 4, 128, 2, 150, 24, 2, "random"),    # 12 query heads per key/value head
    ("dense", 4, 64, 2, 129, 2, 2, "cyclic"),
    ("star", 8, 64, 2, 300, 2, 2, "random"),      # m = 8
    ("star", 1, 128, 2, 65, 2, 2, "cyclic"),
]


@pytest.mark.parametrize("case", DEC_CASES, ids=_ids)
def test_attn_decode_parity(P, case):
    law, q, D, B, S, H, Hkv, kind = case
    m = D // q
    seed = 3500 + S + q
    Qd, Kc, Vc = dec_inputs(seed, B, S, H, Hkv, D)
    pt = schedule(kind, S, q, seed)
    L = np.random.default_rng([seed, 9]).integers(1, S + 1, B).astype(np.int32)
    L[0] = S
    if B > 1:
        L[1] = 1
    shape = P.AttnShape(B, S, H, Hkv, D, q, law)
    O = gpu_decode(P, shape, pt, L, Qd, Kc, Vc)
    ref = oracle.attn_decode(q, law, m, H, Hkv, pt, L, Qd.exact, Kc.exact, Vc.exact)
    assert rel_fro(to_host(O).reshape(B, H * D), ref) <= TOL_BF16


def test_attn_decode_edge_lengths_and_types(P):
    """cache_len 0 and a query of out-of-range type give zero rows; lengths
    past the capacity count as the capacity; cached keys of an out-of-range
    type are skipped (the oracle sees the cache without them)."""
    import torch
    B, S, H, Hkv, D, q = 6, 200, 2, 1, 64, 2
    Qd, Kc, Vc = dec_inputs(3600, B, S, H, Hkv, D)
    pt = schedule("cyclic", S, q)
    pt_bad = pt.copy()
    badk = np.zeros(S, bool)
    badk[[3, 50, 51, 140]] = True
    pt_bad[badk] = [-1, 2, 9, -3]
    L = np.array([0, S + 50, 120, 1, 141, -4], np.int32)
    shape = P.AttnShape(B, S, H, Hkv, D, q)
    O = to_host(gpu_decode(P, shape, pt_bad, L, Qd, Kc, Vc)).reshape(B, H * D)
    assert np.all(O[0] == 0) and np.all(O[5] == 0)
    # sequence 4: query at position 140, whose type is out of range
    assert np.all(O[4] == 0)
    keep = ~badk
    for b, Lb in [(1, S), (2, 120), (3, 1)]:
        kept = np.nonzero(keep[:Lb])[0]
        Lk = len(kept)
        ref = oracle.attn_decode(q, "star", D // q, H, Hkv, pt[kept], np.array([Lk], np.int32),
                                 Qd.exact[b:b + 1], Kc.exact[b:b + 1, kept], Vc.exact[b:b + 1, kept])
        # the query keeps its own position's type: the last kept position is Lb - 1
        assert kept[-1] == Lb - 1
        assert rel_fro(O[b:b + 1], ref) <= TOL_BF16, b
    # bf16 output is the rounding of the fp32 output
    O32 = gpu_decode(P, shape, pt, np.array([5, 200, 7, 9, 100, 1], np.int32), Qd, Kc, Vc)
    O16 = gpu_decode(P, shape, pt, np.array([5, 200, 7, 9, 100, 1], np.int32), Qd, Kc, Vc,
                     out_dtype=torch.bfloat16)
    assert torch.equal(O16, O32.to(torch.bfloat16))


def test_attn_decode_full_size(P):
    """64 sequences at random positions below 2048 over a cache of 2048,
    12 heads of 64, q = 2: every output row against the oracle."""
    B, S, H, Hkv, D, q = 64, 2048, 12, 12, 64, 2
    Qd, Kc, Vc = dec_inputs(3700, B, S, H, Hkv, D)
    pt = schedule("cyclic", S, q)
    L = (synth.decode_positions(3700, B) + 1).astype(np.int32)
    shape = P.AttnShape(B, S, H, Hkv, D, q)
    O = gpu_decode(P, shape, pt, L, Qd, Kc, Vc)
    ref = oracle.attn_decode(q, "star", D // q, H, Hkv, pt, L, Qd.exact, Kc.exact, Vc.exact)
    assert rel_fro(to_host(O).reshape(B, H * D), ref) <= TOL_BF16


def test_attn_decode_matches_forward_rows(P):
    """A decode step at cache length L reproduces row L - 1 of the forward
    over the same sequence (both kernels against the oracle's forward)."""
    B, S, H, Hkv, D, q = 2, 300, 4, 2, 64, 4
    Q, K, V = inputs(3800, B, S, H, Hkv, D)
    pt = schedule("interval", S, q)
    shape = P.AttnShape(B, S, H, Hkv, D, q, "tensor2")
    ref = oracle.attn_fwd(q, "tensor2", D // q, H, Hkv, B, S, pt, Q.exact, K.exact, V.exact)
    L = np.array([S, 171], np.int32)
    rows = np.array([b * S + L[b] - 1 for b in range(B)])
    Qd = synth.Tensor(raw=Q.raw[rows], exact=Q.exact[rows], dtype="bf16")
    Kc = synth.Tensor(raw=K.raw.reshape(B, S, -1), exact=K.exact.reshape(B, S, -1), dtype="bf16")
    Vc = synth.Tensor(raw=V.raw.reshape(B, S, -1), exact=V.exact.reshape(B, S, -1), dtype="bf16")
    Od = to_host(gpu_decode(P, shape, pt, L, Qd, Kc, Vc)).reshape(B, H * D)
    assert rel_fro(Od, ref[rows]) <= TOL_BF16
