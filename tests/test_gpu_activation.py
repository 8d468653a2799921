"""Element-wise bounds on the device activations, through the C ABI.

The kernels evaluate GELU (erf and tanh forms) and its derivative in fp32
with explicit approximations (the erf form through Abramowitz & Stegun
7.1.28, its derivative through 7.1.26).  A tensor-wide Frobenius bar could
hide a narrow band of error, so these tests push dense grids of
pre-activations through every path that applies an activation and bound the
largest element error against the fp64 oracle's activation (itself pinned in
test_oracle_pins.py):

  * forward epilogue: X holds the grid, W is the identity bank (its
    off-diagonal blocks are zero, so every output is exactly the input), Y
    fp32 = act(z);
  * activation gradient with the fused derivative: dY = 1, W the identity,
    Z_prev holds the grid, dX fp32 = act'(z);
  * decode (the persistent stack and the per-projection kernel): one layer,
    identity up and down banks, no bias or residual, so Y = H = the bf16
    rounding of act(z).

Bounds (the ones the library states): values within 1e-6 + 2^-22 |act(z)|,
derivatives within 1e-6 (erf form) or 5e-6 (tanh form).
"""

import numpy as np
import pytest

import oracle
from helpers import to_host, types_dev

pytestmark = pytest.mark.gpu

VAL_ABS, VAL_REL = 1e-6, 2.0 ** -22
DER_ABS = {"gelu": 1e-6, "gelu_tanh": 5e-6}


@pytest.fixture(scope="module")
def P():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32814_amd as P
    return P


def _f32_grid():
    """Dense fp32 grid over [-12, 12] plus the tails and tiny values."""
    g = np.linspace(-12.0, 12.0, (1 << 20) - 64, dtype=np.float64)
    tails = [-60.0, -40.0, -20.0, -16.0, -13.5, 13.5, 16.0, 20.0, 40.0, 60.0, 0.0, -0.0,
             1e-3, -1e-3, 1e-8, -1e-8, 1e-30, -1e-30]
    z = np.concatenate([g, tails, np.zeros(64 - len(tails))]).astype(np.float32)
    return z


def _bf16_values(limit=64.0):
    """Every finite bf16 value of magnitude below `limit` (bit patterns)."""
    import torch
    pos = np.arange(0, 0x7F80, dtype=np.int32).astype(np.int16)
    v = torch.from_numpy(pos).view(torch.bfloat16).to(torch.float32).numpy()
    v = v[np.abs(v) < limit]
    return np.concatenate([v, -v[v > 0]])


def _grid_tensor(z, K, dtype):
    """Pads z to a multiple of K and shapes it [M, K] on the device."""
    import torch
    M = -(-z.size // K)
    a = np.zeros(M * K, np.float32)
    a[:z.size] = z
    t = torch.from_numpy(a.reshape(M, K)).to("cuda")
    return t.to(dtype) if dtype != torch.float32 else t


def _identity_alg(P, K):
    return P.Algebra.equal(2, K, K)


def _check_values(got, z, act):
    ref = oracle.act(act, z.astype(np.float64))
    err = np.abs(got - ref)
    bound = VAL_ABS + VAL_REL * np.abs(ref)
    worst = int(np.argmax(err - bound))
    assert np.all(err <= bound), (f"{act}: error {err[worst]:.3e} at z = {z[worst]!r} "
                                  f"exceeds {bound[worst]:.3e}")


def _check_derivs(got, z, act):
    ref = oracle.act_grad(act, z.astype(np.float64))
    err = np.abs(got - ref)
    worst = int(np.argmax(err))
    assert err.max() <= DER_ABS[act], f"{act}': error {err[worst]:.3e} at z = {z[worst]!r}"


@pytest.mark.parametrize("act", ["gelu", "gelu_tanh"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_forward_epilogue_activation_bound(P, act, dtype):
    import torch
    K = 256
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    z = _f32_grid() if dtype == "f32" else _bf16_values()
    X = _grid_tensor(z, K, td)
    zx = to_host(X).reshape(-1)[:z.size]  # the values the kernel reads
    M = X.shape[0]
    W = torch.eye(K, dtype=td, device="cuda")
    t = types_dev(np.arange(M) % 2)
    Y = P.star_proj_fwd(_identity_alg(P, K), t, X, W, None, act, out_dtype=torch.float32)
    torch.cuda.synchronize()
    _check_values(to_host(Y).reshape(-1)[:z.size], zx, act)


@pytest.mark.parametrize("act", ["gelu", "gelu_tanh"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_activation_gradient_derivative_bound(P, act, dtype):
    import torch
    K = 256
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    z = _f32_grid() if dtype == "f32" else _bf16_values()
    Zp = _grid_tensor(z, K, td)
    zx = to_host(Zp).reshape(-1)[:z.size]
    M = Zp.shape[0]
    W = torch.eye(K, dtype=td, device="cuda")
    dY = torch.ones((M, K), dtype=td, device="cuda")
    t = types_dev(np.arange(M) % 2)
    dX = P.star_proj_bwd_data(_identity_alg(P, K), t, dY, W, Z_prev=Zp, act_prev=act,
                              out_dtype=torch.float32)
    torch.cuda.synchronize()
    _check_derivs(to_host(dX).reshape(-1)[:z.size], zx, act)


@pytest.mark.parametrize("act", ["gelu", "gelu_tanh"])
@pytest.mark.parametrize("width", [256, 1024])
def test_decode_activation_bound(P, act, width):
    """width 256 runs in the persistent stack, width 1024 at 64 rows in the
    per-projection kernel.  H is stored in bf16, so each output must be the
    bf16 rounding of a value within the bound of act(z)."""
    import torch
    M, D = 64, width
    z = _bf16_values()
    per = M * D
    up = P.Algebra.equal(2, D, D)
    dn = P.Algebra.equal(2, D, D)
    W = torch.eye(D, dtype=torch.bfloat16, device="cuda")
    for c0 in range(0, z.size, per):
        zc = z[c0:c0 + per]
        X = _grid_tensor(zc, D, torch.bfloat16)
        if X.shape[0] < M:
            X = torch.cat([X, torch.zeros((M - X.shape[0], D), dtype=torch.bfloat16, device="cuda")])
        zx = to_host(X).reshape(-1)[:zc.size]
        t = types_dev(np.arange(M) % 2)
        Y = P.star_decode(up, dn, t, X, [W], None, [W], None, act, False, out_dtype=torch.float32)
        torch.cuda.synchronize()
        got = to_host(Y).reshape(-1)[:zc.size]
        ref = oracle.act(act, zx.astype(np.float64))
        eps = VAL_ABS + VAL_REL * np.abs(ref)
        # rounding to bf16 is monotone: a value within eps of act(z) rounds
        # to something between the roundings of act(z) - eps and act(z) + eps
        ok = (oracle.round_bf16(ref - eps) <= got) & (got <= oracle.round_bf16(ref + eps))
        bad = np.nonzero(~ok)[0]
        assert bad.size == 0, (f"{act} decode: z = {zx[bad[0]]!r} gave {got[bad[0]]!r}, "
                               f"act(z) = {ref[bad[0]]!r}")
