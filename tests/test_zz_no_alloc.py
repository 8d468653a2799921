"""star_decode_noalloc, the decode step on the library's static workspace,
against star_decode on a workspace of its own: the same kernels on the same
inputs, so the outputs must be bitwise equal.  Calls follow each other on
one stream with shrinking inputs (the static buffer keeps the previous
call's contents, so each call must clear what has to start at zero), and
cover the three decode kernels: the counter stack, the resident stack
(M <= 2) and the per-projection kernel (more layers than the stack holds).
"""

import numpy as np
import pytest

import synth
from helpers import f32_dev, to_dev, types_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32814_amd as P
    return P


def _layers(seed, D, F, L):
    Wu = [to_dev(synth.gaussian(seed, 10 + l, (D, F), 0.02, "bf16")) for l in range(L)]
    Wd = [to_dev(synth.gaussian(seed, 100 + l, (F, D), 0.02, "bf16")) for l in range(L)]
    bu = [f32_dev(synth.gaussian(seed, 200 + l, (F,), 0.02, "f32").exact) for l in range(L)]
    bd = [f32_dev(synth.gaussian(seed, 300 + l, (D,), 0.02, "f32").exact) for l in range(L)]
    return Wu, bu, Wd, bd


def test_noalloc_decode_matches_decode_on_successive_calls(P):
    import torch
    q = 2
    D, F, L = 768, 3072, 12
    up, dn = P.Algebra.equal(q, D, F), P.Algebra.equal(q, F, D)
    Wu, bu, Wd, bd = _layers(1500, D, F, L)
    small_up, small_dn = P.Algebra.equal(q, 128, 256), P.Algebra.equal(q, 256, 128)
    sWu, sbu, sWd, sbd = _layers(1501, 128, 256, 33)
    status = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    # (algebras, weights, M): 64 rows, then 8 (counter stack), 2 and 1
    # (resident stack), then 5 rows through 33 layers (per-projection kernel)
    cases = [((up, dn), (Wu, bu, Wd, bd), 64), ((up, dn), (Wu, bu, Wd, bd), 8),
             ((up, dn), (Wu, bu, Wd, bd), 2), ((up, dn), (Wu, bu, Wd, bd), 1),
             ((small_up, small_dn), (sWu, sbu, sWd, sbd), 5)]
    outs, refs = [], []
    for k, ((u, d), (wu, b_u, wd, b_d), M) in enumerate(cases):
        X = to_dev(synth.gaussian(1502, k, (M, u.K), 1.0, "bf16"))
        t = types_dev((synth.decode_positions(1503 + k, M) % q).astype(np.int32))
        outs.append((P.star_decode_noalloc(u, d, t, X, wu, b_u, wd, b_d, "gelu", True,
                                           out_dtype=torch.float32, status=status), k))
        torch.cuda.synchronize()
        assert int(status.item()) == 0, f"call {k}: a wait bound was hit"
        refs.append(P.star_decode(u, d, t, X, wu, b_u, wd, b_d, "gelu", True, out_dtype=torch.float32))
    # and the first shape once more after the others, without a status word
    X = to_dev(synth.gaussian(1502, 0, (64, D), 1.0, "bf16"))
    t = types_dev((synth.decode_positions(1503, 64) % q).astype(np.int32))
    again = P.star_decode_noalloc(up, dn, t, X, Wu, bu, Wd, bd, "gelu", True, out_dtype=torch.float32)
    torch.cuda.synchronize()
    for (y, k), ref in zip(outs, refs):
        assert torch.equal(y, ref), f"call {k} differs from star_decode"
    assert torch.equal(again, refs[0])


def test_noalloc_decode_argument_errors(P):
    """Host-side checks happen before the static buffer is touched."""
    import ctypes
    V = ctypes.c_void_p
    up, dn = P.Algebra.equal(2, 64, 128), P.Algebra.equal(2, 128, 64)
    arr = (V * 1)(V(16))
    lib = P.binding.LIB
    # 65 rows: more than the decode kernels take
    assert lib.star_decode_noalloc(up.ref, dn.ref, 1, 65, V(16), V(16), 1, arr, None, arr, None, 1, 1,
                                   V(16), 1, None, None) == 6
    # a misaligned status word
    assert lib.star_decode_noalloc(up.ref, dn.ref, 1, 4, V(16), V(16), 1, arr, None, arr, None, 1, 1,
                                   V(16), 1, V(18), None) == 4
    # X must be bfloat16
    assert lib.star_decode_noalloc(up.ref, dn.ref, 1, 4, V(16), V(16), 0, arr, None, arr, None, 1, 1,
                                   V(16), 1, None, None) == 3
