"""CPU fp64 oracle for the row-typed projection Y = X *_q W.

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
library never loads it, and it imports nothing from the product package.

The arithmetic lives in ``star_oracle.c`` (plain fp64 loops, OpenMP over
rows).  This module marshals numpy arrays into it and composes the
multi-projection cases (FFN, training step, decode stack) from the single
projection, mirroring every tensor that the GPU path stores in bfloat16
between two products (rounding to nearest even).

Conventions (Sec. 4 of the paper): X is M x K, W is K x N (input groups are
row blocks of W, output groups column blocks), groups are contiguous in index
order, row types are 0-based.  Law ``"star"`` is the complete-graph algebra
Q_q with B(i,j) = {i,j}; law ``"dense"`` is the ordinary product; law
``"tensor2"`` is the tensor power Q_2^{(x)L} (q = 2^L, appendix "The
Tensor-Square Candidate"): a type-a row reaches input group b for output group
d when every bit of b equals that bit of a or of d (L = 2: the pilot's
36-product law); law ``"graph"`` is the graph algebra Q_G of a directed graph
on the q groups (Sec. "Graph Products with Exact Cost"), given as ``edges``, a
q x q 0/1 matrix (edges[i][j] = 1 for the edge i -> j, diagonal ignored): a
type-i row's slots are its vertex slot i and the edge slots (i, j) of its
out-edges, B(i,i) = {i}, B(i,j) = {i, j} for an edge and empty for a non-edge.
"""

from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "star_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

LAWS = {"star": 0, "dense": 1, "tensor2": 2, "graph": 3}
ACTS = {"none": 0, "gelu": 1, "gelu_tanh": 2, "silu": 3}


def build(force: bool = False) -> str:
    """Compile ``star_oracle.c`` into ``liboracle.so`` (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        i64p = ctypes.POINTER(ctypes.c_int64)
        i32p = ctypes.POINTER(ctypes.c_int32)
        f64p = ctypes.POINTER(ctypes.c_double)
        i64, i32, f64 = ctypes.c_int64, ctypes.c_int, ctypes.c_double
        u8p = ctypes.POINTER(ctypes.c_uint8)
        lib.oracle_proj_fwd.restype = i64
        lib.oracle_proj_fwd.argtypes = [i32, i64p, i64p, i32, u8p, i64, i32p, f64p, f64p,
                                        f64p, i32, f64p, f64p, i64p]
        lib.oracle_proj_bwd_data.restype = i32
        lib.oracle_proj_bwd_data.argtypes = [i32, i64p, i64p, i32, u8p, i64, i32p, f64p,
                                             f64p, f64p, i32, f64p]
        lib.oracle_proj_bwd_weight.restype = i32
        lib.oracle_proj_bwd_weight.argtypes = [i32, i64p, i64p, i32, u8p, i64, i32p, f64p,
                                               f64p, f64p, f64p]
        lib.oracle_bwd_weight_entries.restype = i32
        lib.oracle_bwd_weight_entries.argtypes = [i32, i64p, i64p, i32, u8p, i64, i32p,
                                                  f64p, f64p, i64, i64p, i64p, f64p]
        lib.oracle_round_bf16.restype = f64
        lib.oracle_round_bf16.argtypes = [f64]
        lib.oracle_round_bf16_array.restype = None
        lib.oracle_round_bf16_array.argtypes = [i64, f64p, f64p]
        lib.oracle_act.restype = f64
        lib.oracle_act.argtypes = [i32, f64]
        lib.oracle_act_grad.restype = f64
        lib.oracle_act_grad.argtypes = [i32, f64]
        lib.oracle_products_per_type.restype = i64
        lib.oracle_products_per_type.argtypes = [i32, u8p, i32, i32]
        lib.oracle_row_macs.restype = i64
        lib.oracle_row_macs.argtypes = [i32, u8p, i32, i64p, i64p, i32]
        lib.oracle_square_star.restype = None
        lib.oracle_square_star.argtypes = [i32, i64, f64p, f64p, f64p]
        lib.oracle_square_law.restype = None
        lib.oracle_square_law.argtypes = [i32, u8p, i32, i64, f64p, f64p, f64p]
        lib.oracle_num_threads.restype = i32
        lib.oracle_num_threads.argtypes = []
        lib.oracle_in_support.restype = i32
        lib.oracle_in_support.argtypes = [i32, u8p, i32, i32, i32, i32]
        lib.oracle_attn_in_group.restype = i32
        lib.oracle_attn_in_group.argtypes = [i32, i32, i32, i32]
        lib.oracle_attn_fwd.restype = i32
        lib.oracle_attn_fwd.argtypes = [i32, i32, i64, i32, i32, i64, i64, i32p, f64p, f64p, f64p, f64p, f64p]
        lib.oracle_attn_decode.restype = i32
        lib.oracle_attn_decode.argtypes = [i32, i32, i64, i32, i32, i64, i64, i32p, i32p, f64p, f64p, f64p,
                                           f64p]
        _lib = lib
    return _lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct)) if a is not None else None


@dataclasses.dataclass(frozen=True)
class Alg:
    """An algebra layout: q groups, input widths s, output widths r, law."""

    q: int
    s: tuple
    r: tuple
    law: str = "star"
    edges: tuple = None  # law "graph": q x q 0/1 rows, edges[i][j] for i -> j

    @staticmethod
    def equal(q: int, K: int, N: int, law: str = "star", edges=None) -> "Alg":
        return Alg(q, (K // q,) * q, (N // q,) * q, law, _edge_tuple(edges))

    @property
    def K(self) -> int:
        return int(sum(self.s))

    @property
    def N(self) -> int:
        return int(sum(self.r))

    def _arrays(self):
        return (np.asarray(self.s, dtype=np.int64), np.asarray(self.r, dtype=np.int64))


def _edge_tuple(edges):
    if edges is None:
        return None
    return tuple(tuple(int(bool(v)) for v in row) for row in edges)


def _edges(law: str, q: int, edges):
    """The q x q edge bytes for law "graph" (None for the other laws)."""
    if law != "graph":
        return None
    if edges is None:
        raise ValueError('law "graph" needs edges')
    e = np.ascontiguousarray(np.asarray(edges, dtype=np.uint8).reshape(q, q))
    return e


def _alg_edges(alg: Alg):
    return _edges(alg.law, alg.q, alg.edges)


def num_threads() -> int:
    """OpenMP threads the oracle's loops run on."""
    return int(_load().oracle_num_threads())


def in_support(law: str, i: int, j: int, k: int, q: int = 64, edges=None) -> bool:
    e = _edges(law, q, edges)
    return bool(_load().oracle_in_support(LAWS[law], _p(e, ctypes.c_uint8), q, i, j, k))


def products_per_type(law: str, q: int, i: int, edges=None) -> int:
    e = _edges(law, q, edges)
    return int(_load().oracle_products_per_type(LAWS[law], _p(e, ctypes.c_uint8), q, i))


def row_macs(alg: Alg, i: int) -> int:
    s, r = alg._arrays()
    e = _alg_edges(alg)
    return int(_load().oracle_row_macs(LAWS[alg.law], _p(e, ctypes.c_uint8), alg.q, _p(s, ctypes.c_int64),
                                       _p(r, ctypes.c_int64), i))


def round_bf16(x) -> np.ndarray:
    """Nearest bfloat16 value (ties to even) of each element, as float64."""
    x = _f64(x)
    y = np.empty_like(x)
    _load().oracle_round_bf16_array(x.size, _p(x, ctypes.c_double), _p(y, ctypes.c_double))
    return y


def act(kind: str, z) -> np.ndarray:
    lib = _load()
    z = _f64(z)
    return np.vectorize(lambda v: lib.oracle_act(ACTS[kind], float(v)), otypes=[np.float64])(z)


def act_grad(kind: str, z) -> np.ndarray:
    lib = _load()
    z = _f64(z)
    return np.vectorize(lambda v: lib.oracle_act_grad(ACTS[kind], float(v)), otypes=[np.float64])(z)


def _types(t, M):
    t = np.ascontiguousarray(t, dtype=np.int32)
    if t.shape != (M,):
        raise ValueError("row types must have shape (M,)")
    return t


def proj_fwd(alg: Alg, t, X, W, bias=None, act: str = "none", want_z: bool = False):
    """Alg. 1 plus bias and activation.

    Returns ``(Y, Z, macs, products_per_type)``; ``Z`` is the pre-activation
    (``None`` unless ``want_z``).
    """
    X, W = _f64(X), _f64(W)
    M = X.shape[0]
    t = _types(t, M)
    assert X.shape == (M, alg.K) and W.shape == (alg.K, alg.N)
    s, r = alg._arrays()
    Y = np.empty((M, alg.N), dtype=np.float64)
    Z = np.empty((M, alg.N), dtype=np.float64) if want_z else None
    b = _f64(bias) if bias is not None else None
    ppt = np.zeros(alg.q, dtype=np.int64)
    macs = _load().oracle_proj_fwd(alg.q, _p(s, ctypes.c_int64), _p(r, ctypes.c_int64),
                                   LAWS[alg.law], _p(_alg_edges(alg), ctypes.c_uint8), M,
                                   _p(t, ctypes.c_int32),
                                   _p(X, ctypes.c_double), _p(W, ctypes.c_double),
                                   _p(b, ctypes.c_double), ACTS[act],
                                   _p(Z, ctypes.c_double), _p(Y, ctypes.c_double),
                                   _p(ppt, ctypes.c_int64))
    if macs < 0:
        raise ValueError("row type out of range")
    return Y, Z, int(macs), ppt


def proj_bwd_data(alg: Alg, t, dY, W, Zprev=None, act_prev: str = "none"):
    """Activation gradient (eqs. vjp-xi, vjp-xj), times act'(Zprev) if given."""
    dY, W = _f64(dY), _f64(W)
    M = dY.shape[0]
    t = _types(t, M)
    assert dY.shape == (M, alg.N) and W.shape == (alg.K, alg.N)
    s, r = alg._arrays()
    dX = np.empty((M, alg.K), dtype=np.float64)
    zp = _f64(Zprev) if Zprev is not None else None
    if zp is not None:
        assert zp.shape == (M, alg.K)
    rc = _load().oracle_proj_bwd_data(alg.q, _p(s, ctypes.c_int64), _p(r, ctypes.c_int64),
                                      LAWS[alg.law], _p(_alg_edges(alg), ctypes.c_uint8), M,
                                   _p(t, ctypes.c_int32),
                                      _p(dY, ctypes.c_double), _p(W, ctypes.c_double),
                                      _p(zp, ctypes.c_double), ACTS[act_prev],
                                      _p(dX, ctypes.c_double))
    if rc:
        raise ValueError("row type out of range")
    return dX


def proj_bwd_weight(alg: Alg, t, X, dY):
    """Weight and bias gradients (eqs. vjp-wii, vjp-wij, vjp-wjj)."""
    X, dY = _f64(X), _f64(dY)
    M = X.shape[0]
    t = _types(t, M)
    assert X.shape == (M, alg.K) and dY.shape == (M, alg.N)
    s, r = alg._arrays()
    dW = np.empty((alg.K, alg.N), dtype=np.float64)
    db = np.empty(alg.N, dtype=np.float64)
    rc = _load().oracle_proj_bwd_weight(alg.q, _p(s, ctypes.c_int64), _p(r, ctypes.c_int64),
                                        LAWS[alg.law], _p(_alg_edges(alg), ctypes.c_uint8), M,
                                   _p(t, ctypes.c_int32),
                                        _p(X, ctypes.c_double), _p(dY, ctypes.c_double),
                                        _p(dW, ctypes.c_double), _p(db, ctypes.c_double))
    if rc:
        raise ValueError("row type out of range")
    return dW, db


def bwd_weight_entries(alg: Alg, t, X, dY, kk, nn):
    """Selected entries dW[kk[e], nn[e]], each summed over the whole batch."""
    X, dY = _f64(X), _f64(dY)
    M = X.shape[0]
    t = _types(t, M)
    kk = np.ascontiguousarray(kk, dtype=np.int64)
    nn = np.ascontiguousarray(nn, dtype=np.int64)
    s, r = alg._arrays()
    out = np.empty(kk.size, dtype=np.float64)
    rc = _load().oracle_bwd_weight_entries(alg.q, _p(s, ctypes.c_int64), _p(r, ctypes.c_int64),
                                           LAWS[alg.law], _p(_alg_edges(alg), ctypes.c_uint8), M,
                                   _p(t, ctypes.c_int32),
                                           _p(X, ctypes.c_double), _p(dY, ctypes.c_double),
                                           kk.size, _p(kk, ctypes.c_int64), _p(nn, ctypes.c_int64),
                                           _p(out, ctypes.c_double))
    if rc:
        raise ValueError("row type out of range")
    return out


def square_star(q: int, bs: int, A, B) -> np.ndarray:
    """Square-rule product of q x q block arrays (eqs. q-product-diag/-off)."""
    A, B = _f64(A), _f64(B)
    n = q * bs
    assert A.shape == (n, n) and B.shape == (n, n)
    C = np.empty((n, n), dtype=np.float64)
    _load().oracle_square_star(q, bs, _p(A, ctypes.c_double), _p(B, ctypes.c_double),
                               _p(C, ctypes.c_double))
    return C


def square_law(law: str, q: int, bs: int, A, B, edges=None) -> np.ndarray:
    """Row-column rule with the law's support: (A*B)_ij = sum over k in
    B(i,j) of A_ik B_kj, for q x q block arrays of b x b blocks."""
    A, B = _f64(A), _f64(B)
    n = q * bs
    assert A.shape == (n, n) and B.shape == (n, n)
    C = np.empty((n, n), dtype=np.float64)
    e = _edges(law, q, edges)
    _load().oracle_square_law(LAWS[law], _p(e, ctypes.c_uint8), q, bs, _p(A, ctypes.c_double),
                              _p(B, ctypes.c_double), _p(C, ctypes.c_double))
    return C


# ---- compositions ----------------------------------------------------------


def ffn_fwd(up: Alg, down: Alg, t, X, W_up, b_up, W_down, b_down, act: str = "gelu",
            mirror_bf16: bool = True):
    """Two-map FFN with the same row types on both projections (Sec. 4,
    "Projection Shapes"; Sec. 5.2).

    Z = X *W_up + b_up;  H = act(Z);  Y = H * W_down + b_down.
    With ``mirror_bf16`` the hidden H and the saved pre-activation Z are
    rounded to bfloat16, as the GPU path stores them.  Returns (Z, H, Y).
    """
    H, Z, _, _ = proj_fwd(up, t, X, W_up, b_up, act, want_z=True)
    if mirror_bf16:
        H = round_bf16(H)
        Z = round_bf16(Z)
    Y, _, _, _ = proj_fwd(down, t, H, W_down, b_down, "none")
    return Z, H, Y


def ffn_bwd(up: Alg, down: Alg, t, X, Z, H, W_up, W_down, dY, act: str = "gelu",
            mirror_bf16: bool = True):
    """Backward of ``ffn_fwd`` (App. "Vector--Jacobian Products", chained).

    dZ = (dY *^T W_down) . act'(Z);  dX = dZ *^T W_up;
    dW_down, db_down from (H, dY);  dW_up, db_up from (X, dZ).
    With ``mirror_bf16`` the stored dZ is rounded to bfloat16.
    Returns dict of dX, dZ, dW_up, db_up, dW_down, db_down.
    """
    dZ = proj_bwd_data(down, t, dY, W_down, Zprev=Z, act_prev=act)
    if mirror_bf16:
        dZ = round_bf16(dZ)
    dX = proj_bwd_data(up, t, dZ, W_up)
    dW_down, db_down = proj_bwd_weight(down, t, H, dY)
    dW_up, db_up = proj_bwd_weight(up, t, X, dZ)
    return dict(dX=dX, dZ=dZ, dW_up=dW_up, db_up=db_up, dW_down=dW_down, db_down=db_down)


def swiglu_ffn_fwd(up: Alg, down: Alg, t, X, W_gate, b_gate, W_up, b_up, W_down, b_down,
                   mirror_bf16: bool = True):
    """Gated FFN (SwiGLU) with the same row types on all three projections:
    Z_g = X * W_gate + b_gate;  Z_u = X * W_up + b_up;
    H = silu(Z_g) . Z_u;  Y = H * W_down + b_down.
    Gate and up are two projections of the same layout ``up``.  With
    ``mirror_bf16`` Z_g, Z_u and H are rounded to bfloat16, as the GPU path
    stores them.  Returns (Z_g, Z_u, H, Y)."""
    Zg, _, _, _ = proj_fwd(up, t, X, W_gate, b_gate, "none")
    Zu, _, _, _ = proj_fwd(up, t, X, W_up, b_up, "none")
    if mirror_bf16:
        Zg, Zu = round_bf16(Zg), round_bf16(Zu)
    H = act("silu", Zg) * Zu
    if mirror_bf16:
        H = round_bf16(H)
    Y, _, _, _ = proj_fwd(down, t, H, W_down, b_down, "none")
    return Zg, Zu, H, Y


def swiglu_ffn_bwd(up: Alg, down: Alg, t, X, Zg, Zu, H, W_gate, W_up, W_down, dY,
                   mirror_bf16: bool = True):
    """Backward of ``swiglu_ffn_fwd``:
    dH = dY *^T W_down;  dZ_g = dH . Z_u . silu'(Z_g);  dZ_u = dH . silu(Z_g);
    dX = dZ_g *^T W_gate + dZ_u *^T W_up;  dW_gate, db_gate from (X, dZ_g);
    dW_up, db_up from (X, dZ_u);  dW_down, db_down from (H, dY).
    With ``mirror_bf16`` the stored dH, dZ_g and dZ_u are rounded to
    bfloat16.  Returns a dict of the gradients and dZ_g, dZ_u."""
    dH = proj_bwd_data(down, t, dY, W_down)
    if mirror_bf16:
        dH = round_bf16(dH)
    dZg = dH * Zu * act_grad("silu", Zg)
    dZu = dH * act("silu", Zg)
    if mirror_bf16:
        dZg, dZu = round_bf16(dZg), round_bf16(dZu)
    dX = proj_bwd_data(up, t, dZg, W_gate) + proj_bwd_data(up, t, dZu, W_up)
    dW_gate, db_gate = proj_bwd_weight(up, t, X, dZg)
    dW_up, db_up = proj_bwd_weight(up, t, X, dZu)
    dW_down, db_down = proj_bwd_weight(down, t, H, dY)
    return dict(dX=dX, dZ_gate=dZg, dZ_up=dZu, dW_gate=dW_gate, db_gate=db_gate, dW_up=dW_up,
                db_up=db_up, dW_down=dW_down, db_down=db_down)


def decode_stack(up: Alg, down: Alg, t, X, W_ups, b_ups, W_downs, b_downs,
                 act: str = "gelu", residual: bool = True, mirror_bf16: bool = True):
    """FFN stack for one decode step: h <- h + FFN_l(h), l = 1..L (Sec. 5.3).

    Each layer's projection input is the bfloat16 rounding of the running
    state h (mirrored when ``mirror_bf16``), H is stored in bfloat16, and h
    itself is carried at full precision.  Without ``residual`` the layer
    output replaces h.  Returns the final h.
    """
    h = _f64(X)
    for Wu, bu, Wd, bd in zip(W_ups, b_ups, W_downs, b_downs):
        a = round_bf16(h) if mirror_bf16 else h
        _, _, f = ffn_fwd(up, down, t, a, Wu, bu, Wd, bd, act, mirror_bf16)
        h = h + f if residual else f
    return h


def decode_stack_gated(up: Alg, down: Alg, t, X, W_gates, b_gates, W_ups, b_ups, W_downs, b_downs,
                       residual: bool = True, mirror_bf16: bool = True):
    """Gated-FFN (SwiGLU) stack for one decode step:
    h <- h + (silu(a W_gate + b_gate) . (a W_up + b_up)) W_down + b_down with
    a the bfloat16 rounding of h; the hidden H is stored in bfloat16, h is
    carried at full precision (the pre-activations stay in fp32, as the GPU
    stack keeps them in registers).  Returns the final h."""
    h = _f64(X)
    for Wg, bg, Wu, bu, Wd, bd in zip(W_gates, b_gates, W_ups, b_ups, W_downs, b_downs):
        a = round_bf16(h) if mirror_bf16 else h
        Zg, _, _, _ = proj_fwd(up, t, a, Wg, bg, "none")
        Zu, _, _, _ = proj_fwd(up, t, a, Wu, bu, "none")
        H = act("silu", Zg) * Zu
        if mirror_bf16:
            H = round_bf16(H)
        f, _, _, _ = proj_fwd(down, t, H, Wd, bd, "none")
        h = h + f if residual else f
    return h


# ---- algebraic attention ------------------------------------------------------


def attn_in_group(law: str, i: int, j: int, a: int) -> bool:
    """Whether feature group a is in F(i, j) (eqs. feature-set,
    tensor-square-feature-set)."""
    return bool(_load().oracle_attn_in_group(LAWS[law], i, j, a))


def attn_fwd(q: int, law: str, m: int, n_heads: int, n_kv: int, B: int, S: int, pos_type, Q, K, V,
             want_lse: bool = False):
    """Causal attention with the algebraic score (Alg. attention-training,
    forward): Q [B S, n_heads q m], K and V [B S, n_kv q m], token-major;
    pos_type[p] is the type of position p.  Returns O like Q, and with
    ``want_lse`` also the natural log of each query's softmax denominator
    [B, n_heads, S]."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    pt = np.ascontiguousarray(pos_type, dtype=np.int32)
    dh = q * m
    assert Q.shape == (B * S, n_heads * dh) and K.shape == (B * S, n_kv * dh) and V.shape == K.shape
    assert pt.shape == (S,)
    O = np.empty_like(Q)
    lse = np.empty((B, n_heads, S), np.float64) if want_lse else None
    st = _load().oracle_attn_fwd(q, LAWS[law], m, n_heads, n_kv, B, S, _p(pt, ctypes.c_int32), _p(Q, ctypes.c_double),
                                 _p(K, ctypes.c_double), _p(V, ctypes.c_double), _p(O, ctypes.c_double),
                                 _p(lse, ctypes.c_double) if want_lse else None)
    if st != 0:
        raise ValueError("bad attention arguments (type out of range or head counts)")
    return (O, lse) if want_lse else O


def attn_decode(q: int, law: str, m: int, n_heads: int, n_kv: int, pos_type, cache_len, Q, K_cache, V_cache):
    """One decode step (Alg. attention-decoding): Q [B, n_heads q m]; the
    caches [B, S_max, n_kv q m] hold cache_len[b] positions of sequence b,
    whose query is at position cache_len[b] - 1.  Returns O [B, n_heads q m]."""
    Q, Kc, Vc = _f64(Q), _f64(K_cache), _f64(V_cache)
    pt = np.ascontiguousarray(pos_type, dtype=np.int32)
    cl = np.ascontiguousarray(cache_len, dtype=np.int32)
    B, S_max = Kc.shape[0], Kc.shape[1]
    dh = q * m
    assert Q.shape == (B, n_heads * dh) and Kc.shape == (B, S_max, n_kv * dh) and Vc.shape == Kc.shape
    assert pt.shape == (S_max,) and cl.shape == (B,)
    O = np.empty_like(Q)
    st = _load().oracle_attn_decode(q, LAWS[law], m, n_heads, n_kv, B, S_max, _p(pt, ctypes.c_int32),
                                    _p(cl, ctypes.c_int32), _p(Q, ctypes.c_double), _p(Kc, ctypes.c_double),
                                    _p(Vc, ctypes.c_double), _p(O, ctypes.c_double))
    if st != 0:
        raise ValueError("bad attention arguments")
    return O
