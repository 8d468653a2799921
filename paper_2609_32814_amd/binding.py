"""ctypes binding of libstarq's C ABI (``include/star_proj.h``).

Argument marshalling only: torch tensors supply device pointers, the current
HIP stream, and (when the caller passes none) output and workspace buffers.
Every step of the computation runs in the library's HIP kernels.  Importing
this module fails loudly if ``libstarq.so`` has not been built.
"""

from __future__ import annotations

import ctypes
import os
from typing import Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libstarq.so")

STAR_OK = 0
STATUS_NAMES = {0: "STAR_OK", 1: "STAR_ERR_ARG", 2: "STAR_ERR_SHAPE", 3: "STAR_ERR_DTYPE",
                4: "STAR_ERR_ALIGN", 5: "STAR_ERR_WORKSPACE", 6: "STAR_ERR_UNSUPPORTED",
                7: "STAR_ERR_HIP"}
DTYPES = {torch.float32: 0, torch.bfloat16: 1}
ACTS = {"none": 0, "gelu": 1, "gelu_tanh": 2}
LAWS = {"star": 0, "dense": 1, "tensor2": 2, "graph": 3}
OPS = {"fwd": 0, "bwd_data": 1, "bwd_weight": 2, "ffn_fwd": 3, "decode": 4}
MAX_Q = 64


class StarError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} "
                         f"({star_status_string(status)})")


class _CAlgebra(ctypes.Structure):
    _fields_ = [("q", ctypes.c_int32), ("s", ctypes.POINTER(ctypes.c_int64)),
                ("r", ctypes.POINTER(ctypes.c_int64)), ("law", ctypes.c_int),
                ("edges", ctypes.POINTER(ctypes.c_uint8))]


class _CAttnShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("seq_len", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("q", ctypes.c_int32),
                ("law", ctypes.c_int)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2609_32814_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    A = ctypes.POINTER(_CAlgebra)
    i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    E = ctypes.c_int
    lib.star_proj_fwd.argtypes = [A, i64, P, P, E, P, E, P, E, P, P, E, P, sz, P]
    lib.star_proj_bwd_data.argtypes = [A, i64, P, P, E, P, E, P, E, P, E, P, sz, P]
    lib.star_proj_bwd_weight.argtypes = [A, i64, P, P, E, P, E, P, P, P, sz, P]
    lib.star_ffn_fwd.argtypes = [A, A, i64, P, P, P, P, P, P, E, P, P, P, E, E, P, sz, P]
    lib.star_decode.argtypes = [A, A, i32, i64, P, P, E, ctypes.POINTER(P), ctypes.POINTER(P),
                                ctypes.POINTER(P), ctypes.POINTER(P), E, i32, P, E, P, sz, P]
    lib.star_decode_gated.argtypes = [A, A, i32, i64, P, P, E, ctypes.POINTER(P), ctypes.POINTER(P),
                                      ctypes.POINTER(P), ctypes.POINTER(P), ctypes.POINTER(P),
                                      ctypes.POINTER(P), i32, P, E, P, sz, P]
    lib.star_decode_status.argtypes = [P, sz, ctypes.POINTER(i32), P]
    lib.star_decode_noalloc.argtypes = [A, A, i32, i64, P, P, E, ctypes.POINTER(P), ctypes.POINTER(P),
                                        ctypes.POINTER(P), ctypes.POINTER(P), E, i32, P, E, P, P]
    lib.star_workspace_bytes.argtypes = [i32, A, A, i64]
    lib.star_workspace_bytes.restype = sz
    lib.star_count_products.argtypes = [A, ctypes.POINTER(i64)]
    lib.star_set_fwd_tiles.argtypes = [ctypes.c_int]
    lib.star_set_fwd_tiles.restype = ctypes.c_int
    lib.star_count_macs.argtypes = [A, ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.star_validate_types.argtypes = [i64, P, i32, ctypes.POINTER(i64), P, sz, P]
    lib.star_plan_bytes.argtypes = [i32, i64]
    lib.star_plan_bytes.restype = sz
    lib.star_type_plan.argtypes = [i32, i64, P, P, sz, P]
    lib.star_proj_fwd_planned.argtypes = [A, i64, P, P, E, P, E, P, E, P, P, E, P]
    lib.star_proj_bwd_data_planned.argtypes = [A, i64, P, P, E, P, E, P, E, P, E, P]
    lib.star_proj_bwd_weight_planned.argtypes = [A, i64, P, P, E, P, E, P, P, P, sz, P]
    lib.star_swiglu_fwd.argtypes = [i64, P, P, E, P, P]
    lib.star_swiglu_bwd.argtypes = [i64, P, P, P, E, P, P, P]
    lib.star_add.argtypes = [i64, P, P, E, P, P]
    lib.star_swiglu_merged_fwd.argtypes = [i64, i64, P, E, P, P]
    lib.star_swiglu_up_fwd_planned.argtypes = [A, i64, P, P, E, P, E, P, P, P, E, P]
    S = ctypes.POINTER(_CAttnShape)
    lib.star_attn_fwd.argtypes = [S, P, P, P, P, E, P, E, P, P]
    lib.star_attn_decode_workspace_bytes.argtypes = [S]
    lib.star_attn_decode_workspace_bytes.restype = sz
    lib.star_attn_decode.argtypes = [S, P, P, P, P, P, E, P, E, P, sz, P]
    lib.star_status_string.argtypes = [E]
    lib.star_status_string.restype = ctypes.c_char_p
    for name in ("star_proj_fwd", "star_proj_bwd_data", "star_proj_bwd_weight", "star_ffn_fwd",
                 "star_decode", "star_count_products", "star_count_macs", "star_validate_types",
                 "star_type_plan", "star_proj_fwd_planned", "star_proj_bwd_data_planned",
                 "star_proj_bwd_weight_planned", "star_swiglu_fwd", "star_swiglu_bwd", "star_add",
                 "star_decode_gated", "star_decode_status", "star_decode_noalloc", "star_attn_fwd",
                 "star_attn_decode", "star_swiglu_merged_fwd", "star_swiglu_up_fwd_planned"):
        getattr(lib, name).restype = E
    return lib


LIB = _load()


class Algebra:
    """q groups of input widths ``s`` and output widths ``r`` under a law;
    law ``"graph"`` takes ``edges``, a q x q 0/1 matrix (edges[i][j] for the
    edge i -> j of the graph algebra Q_G; the diagonal is ignored)."""

    def __init__(self, q: int, s: Sequence[int], r: Sequence[int], law: str = "star", edges=None):
        self.q, self.law = int(q), law
        self.s, self.r = tuple(int(v) for v in s), tuple(int(v) for v in r)
        if len(self.s) != self.q or len(self.r) != self.q:
            raise ValueError("s and r need q entries each")
        self.edges = None
        if edges is not None:
            rows = [[int(bool(v)) for v in row] for row in edges]
            if len(rows) != self.q or any(len(row) != self.q for row in rows):
                raise ValueError("edges must be a q x q matrix")
            self.edges = tuple(tuple(row) for row in rows)
        if law == "graph" and self.edges is None:
            raise ValueError('law "graph" needs edges')
        self._s = (ctypes.c_int64 * self.q)(*self.s)
        self._r = (ctypes.c_int64 * self.q)(*self.r)
        self._e = None
        if self.edges is not None:
            self._e = (ctypes.c_uint8 * (self.q * self.q))(*[v for row in self.edges for v in row])
        self._c = _CAlgebra(self.q, ctypes.cast(self._s, ctypes.POINTER(ctypes.c_int64)),
                            ctypes.cast(self._r, ctypes.POINTER(ctypes.c_int64)), LAWS[law],
                            ctypes.cast(self._e, ctypes.POINTER(ctypes.c_uint8)) if self._e is not None
                            else None)

    @classmethod
    def equal(cls, q: int, K: int, N: int, law: str = "star", edges=None) -> "Algebra":
        if K % q or N % q:
            raise ValueError("equal groups need q | K and q | N")
        return cls(q, [K // q] * q, [N // q] * q, law, edges)

    @property
    def K(self) -> int:
        return sum(self.s)

    @property
    def N(self) -> int:
        return sum(self.r)

    @property
    def ref(self):
        return ctypes.byref(self._c)

    def with_law(self, law: str) -> "Algebra":
        return Algebra(self.q, self.s, self.r, law, self.edges)

    def merged_gate_up(self) -> "Algebra":
        """The algebra of the merged gate/up product of this up layout:
        output widths doubled (gate and up of each group side by side)."""
        return Algebra(self.q, self.s, [2 * x for x in self.r], self.law, self.edges)

    def __repr__(self):
        return f"Algebra(q={self.q}, s={self.s}, r={self.r}, law={self.law!r})"


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check(status: int, where: str):
    if status != STAR_OK:
        raise StarError(status, where)


def _dt(t: torch.Tensor) -> int:
    if t.dtype not in DTYPES:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return DTYPES[t.dtype]


def _ws(op: str, alg: Algebra, alg2, M: int, device, ws):
    need = star_workspace_bytes(op, alg, alg2, M)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=device)
    if not ws.is_contiguous() or ws.device != device:
        raise ValueError("ws must be a contiguous buffer on the operands' device")
    return ws, ws.numel() * ws.element_size()


def _need(t, name: str, shape, dtypes=None, device=None):
    """Checks a tensor argument before its pointer crosses the ABI: a device
    tensor of the expected shape and dtype, dense in row-major order (the
    library reads every buffer as a plain row-major array)."""
    if t is None:
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if tuple(t.shape) != tuple(int(v) for v in shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {tuple(dtypes)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous (row-major, no strides)")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    return t


def _gpu(device):
    """Every tensor of a call sits on `device`; it must be a GPU."""
    if torch.device(device).type != "cuda":
        raise ValueError("the library takes GPU tensors only")


def _opt(t, name: str, shape, dtypes=None, device=None):
    return None if t is None else _need(t, name, shape, dtypes, device)


_FLOATS = (torch.float32, torch.bfloat16)
_F32 = (torch.float32,)
_BF16 = (torch.bfloat16,)
_I32 = (torch.int32,)


def _rows(X, name: str, K: int):
    if not isinstance(X, torch.Tensor) or X.dim() != 2:
        raise ValueError(f"{name} must be a 2-D tensor")
    _need(X, name, (X.shape[0], K), _FLOATS)
    return X.shape[0], X.device


def _types(row_type, M: int, device):
    return _need(row_type, "row_type", (M,), _I32, device)


def star_status_string(status: int) -> str:
    return LIB.star_status_string(int(status)).decode()


def star_workspace_bytes(op: str, alg: Algebra, alg2: Algebra | None, M: int) -> int:
    return int(LIB.star_workspace_bytes(OPS[op], alg.ref, alg2.ref if alg2 else None, int(M)))


TILES = {"auto": 0, "wide": 1, "small": 2, "wide192": 3}


def star_set_fwd_tiles(tiles: str) -> str:
    """Forward tile size for bf16 operands: "auto" (by the tiles' fill and
    padding), "wide" (256 x 256), "wide192" (256 x 192 for the star and dense
    laws) or "small" (64 x 128); process-wide.  Returns the previous
    setting."""
    if tiles not in TILES:
        raise ValueError(f"tiles must be one of {sorted(TILES)}, not {tiles!r}")
    prev = int(LIB.star_set_fwd_tiles(TILES[tiles]))
    return {v: k for k, v in TILES.items()}[prev]


def star_count_products(alg: Algebra) -> list[int]:
    out = (ctypes.c_int64 * alg.q)()
    _check(LIB.star_count_products(alg.ref, out), "star_count_products")
    return list(out)


def star_count_macs(alg: Algebra, rows_per_type: Sequence[int]) -> int:
    rows = (ctypes.c_int64 * alg.q)(*[int(v) for v in rows_per_type])
    macs = ctypes.c_int64()
    _check(LIB.star_count_macs(alg.ref, rows, ctypes.byref(macs)), "star_count_macs")
    return int(macs.value)


def star_validate_types(row_type: torch.Tensor, q: int, ws=None) -> int:
    n_bad = ctypes.c_int64()
    _types(row_type, row_type.numel(), row_type.device)
    ws = ws if ws is not None else torch.empty(16, dtype=torch.uint8, device=row_type.device)
    _gpu(row_type.device)
    _check(LIB.star_validate_types(row_type.numel(), _ptr(row_type), int(q), ctypes.byref(n_bad),
                                   _ptr(ws), ws.numel(), _stream(row_type.device)),
           "star_validate_types")
    return int(n_bad.value)


def star_plan_bytes(q: int, M: int) -> int:
    return int(LIB.star_plan_bytes(int(q), int(M)))


def star_type_plan(q: int, row_type: torch.Tensor, plan=None):
    """Builds the type plan of ``row_type`` (device uint8 buffer)."""
    M = row_type.numel()
    dev = row_type.device
    _types(row_type, M, dev)
    if plan is None:
        plan = torch.empty(max(star_plan_bytes(q, M), 16), dtype=torch.uint8, device=dev)
    _need(plan, "plan", tuple(plan.shape), None, dev)
    _gpu(dev)
    _check(LIB.star_type_plan(int(q), M, _ptr(row_type), _ptr(plan), plan.numel(), _stream(dev)),
           "star_type_plan")
    return plan


def star_proj_fwd_planned(alg: Algebra, plan: torch.Tensor, X: torch.Tensor, W: torch.Tensor,
                          bias: torch.Tensor | None = None, act: str = "none", Z_out=None,
                          Y=None, out_dtype=None):
    M, dev = _rows(X, "X", alg.K)
    _need(W, "W", (alg.K, alg.N), (X.dtype,), dev)
    _opt(bias, "bias", (alg.N,), _F32, dev)
    _need(plan, "plan", tuple(plan.shape), None, dev)
    if Y is None:
        Y = torch.empty((M, alg.N), dtype=out_dtype or X.dtype, device=dev)
    _need(Y, "Y", (M, alg.N), _FLOATS, dev)
    want_z = Z_out is not None and Z_out is not False
    if Z_out is True:
        Z_out = torch.empty((M, alg.N), dtype=Y.dtype, device=dev)
    if want_z:
        _need(Z_out, "Z_out", (M, alg.N), (Y.dtype,), dev)
    _gpu(dev)
    _check(LIB.star_proj_fwd_planned(alg.ref, M, _ptr(plan), _ptr(X), _dt(X), _ptr(W), _dt(W),
                                     _ptr(bias), ACTS[act], _ptr(Z_out) if want_z else None,
                                     _ptr(Y), _dt(Y), _stream(dev)), "star_proj_fwd_planned")
    return (Y, Z_out) if want_z else Y


def star_proj_bwd_data_planned(alg: Algebra, plan: torch.Tensor, dY: torch.Tensor,
                               W: torch.Tensor, Z_prev=None, act_prev: str = "none", dX=None,
                               out_dtype=None):
    M, dev = _rows(dY, "dY", alg.N)
    _need(W, "W", (alg.K, alg.N), (dY.dtype,), dev)
    _opt(Z_prev, "Z_prev", (M, alg.K), (dY.dtype,), dev)
    _need(plan, "plan", tuple(plan.shape), None, dev)
    if dX is None:
        dX = torch.empty((M, alg.K), dtype=out_dtype or dY.dtype, device=dev)
    _need(dX, "dX", (M, alg.K), _FLOATS, dev)
    _gpu(dev)
    _check(LIB.star_proj_bwd_data_planned(alg.ref, M, _ptr(plan), _ptr(dY), _dt(dY), _ptr(W),
                                          _dt(W), _ptr(Z_prev), ACTS[act_prev], _ptr(dX),
                                          _dt(dX), _stream(dev)), "star_proj_bwd_data_planned")
    return dX


def star_proj_bwd_weight_planned(alg: Algebra, plan: torch.Tensor, X: torch.Tensor,
                                 dY: torch.Tensor, dW=None, dbias=None, want_dbias: bool = True,
                                 ws=None):
    M, dev = _rows(X, "X", alg.K)
    _need(dY, "dY", (M, alg.N), (X.dtype,), dev)
    _need(plan, "plan", tuple(plan.shape), None, dev)
    if dW is None:
        dW = torch.empty((alg.K, alg.N), dtype=torch.float32, device=dev)
    if dbias is None and want_dbias:
        dbias = torch.empty(alg.N, dtype=torch.float32, device=dev)
    _need(dW, "dW", (alg.K, alg.N), _F32, dev)
    _opt(dbias, "dbias", (alg.N,), _F32, dev)
    _gpu(dev)
    ws, nbytes = _ws("bwd_weight", alg, None, M, dev, ws)
    _check(LIB.star_proj_bwd_weight_planned(alg.ref, M, _ptr(plan), _ptr(X), _dt(X), _ptr(dY),
                                            _dt(dY), _ptr(dW), _ptr(dbias), _ptr(ws), nbytes,
                                            _stream(dev)), "star_proj_bwd_weight_planned")
    return dW, dbias


def star_proj_fwd(alg: Algebra, row_type: torch.Tensor, X: torch.Tensor, W: torch.Tensor,
                  bias: torch.Tensor | None = None, act: str = "none", Z_out=None, Y=None,
                  out_dtype=None, ws=None):
    """Y = act(X *_q W + bias).  ``Z_out=True`` allocates and returns the
    pre-activation too.  Returns Y, or (Y, Z) when Z_out is requested."""
    M, dev = _rows(X, "X", alg.K)
    _types(row_type, M, dev)
    _need(W, "W", (alg.K, alg.N), (X.dtype,), dev)
    _opt(bias, "bias", (alg.N,), _F32, dev)
    out_dtype = out_dtype or X.dtype
    if Y is None:
        Y = torch.empty((M, alg.N), dtype=out_dtype, device=dev)
    _need(Y, "Y", (M, alg.N), _FLOATS, dev)
    want_z = Z_out is not None and Z_out is not False
    if Z_out is True:
        Z_out = torch.empty((M, alg.N), dtype=Y.dtype, device=dev)
    if want_z:
        _need(Z_out, "Z_out", (M, alg.N), (Y.dtype,), dev)
    _gpu(dev)
    ws, nbytes = _ws("fwd", alg, None, M, dev, ws)
    _check(LIB.star_proj_fwd(alg.ref, M, _ptr(row_type), _ptr(X), _dt(X), _ptr(W), _dt(W),
                             _ptr(bias), ACTS[act], _ptr(Z_out) if want_z else None, _ptr(Y),
                             _dt(Y), _ptr(ws), nbytes, _stream(dev)), "star_proj_fwd")
    return (Y, Z_out) if want_z else Y


def star_proj_bwd_data(alg: Algebra, row_type: torch.Tensor, dY: torch.Tensor, W: torch.Tensor,
                       Z_prev: torch.Tensor | None = None, act_prev: str = "none", dX=None,
                       out_dtype=None, ws=None):
    """dX = (dY *_q^T W) [. act_prev'(Z_prev)]."""
    M, dev = _rows(dY, "dY", alg.N)
    _types(row_type, M, dev)
    _need(W, "W", (alg.K, alg.N), (dY.dtype,), dev)
    _opt(Z_prev, "Z_prev", (M, alg.K), (dY.dtype,), dev)
    if dX is None:
        dX = torch.empty((M, alg.K), dtype=out_dtype or dY.dtype, device=dev)
    _need(dX, "dX", (M, alg.K), _FLOATS, dev)
    _gpu(dev)
    ws, nbytes = _ws("bwd_data", alg, None, M, dev, ws)
    _check(LIB.star_proj_bwd_data(alg.ref, M, _ptr(row_type), _ptr(dY), _dt(dY), _ptr(W), _dt(W),
                                  _ptr(Z_prev), ACTS[act_prev], _ptr(dX), _dt(dX), _ptr(ws),
                                  nbytes, _stream(dev)), "star_proj_bwd_data")
    return dX


def star_proj_bwd_weight(alg: Algebra, row_type: torch.Tensor, X: torch.Tensor, dY: torch.Tensor,
                         dW=None, dbias=None, want_dbias: bool = True, ws=None):
    """(dW, dbias) in fp32; dbias is None unless requested."""
    M, dev = _rows(X, "X", alg.K)
    _types(row_type, M, dev)
    _need(dY, "dY", (M, alg.N), (X.dtype,), dev)
    if dW is None:
        dW = torch.empty((alg.K, alg.N), dtype=torch.float32, device=dev)
    if dbias is None and want_dbias:
        dbias = torch.empty(alg.N, dtype=torch.float32, device=dev)
    _need(dW, "dW", (alg.K, alg.N), _F32, dev)
    _opt(dbias, "dbias", (alg.N,), _F32, dev)
    _gpu(dev)
    ws, nbytes = _ws("bwd_weight", alg, None, M, dev, ws)
    _check(LIB.star_proj_bwd_weight(alg.ref, M, _ptr(row_type), _ptr(X), _dt(X), _ptr(dY),
                                    _dt(dY), _ptr(dW), _ptr(dbias), _ptr(ws), nbytes,
                                    _stream(dev)), "star_proj_bwd_weight")
    return dW, dbias


def star_ffn_fwd(up: Algebra, down: Algebra, row_type: torch.Tensor, X: torch.Tensor,
                 W_up: torch.Tensor, b_up, W_down: torch.Tensor, b_down, act: str = "gelu",
                 save_z: bool = True, H=None, Y=None, Z_up=None, out_dtype=None, ws=None):
    """Returns (Z_up or None, H, Y)."""
    M, dev = _rows(X, "X", up.K)
    _types(row_type, M, dev)
    if down.K != up.N or down.N != up.K:
        raise ValueError("down must map the up projection's output back to its input width")
    _need(W_up, "W_up", (up.K, up.N), (X.dtype,), dev)
    _need(W_down, "W_down", (down.K, down.N), (X.dtype,), dev)
    _opt(b_up, "b_up", (up.N,), _F32, dev)
    _opt(b_down, "b_down", (down.N,), _F32, dev)
    if H is None:
        H = torch.empty((M, up.N), dtype=X.dtype, device=dev)
    if Y is None:
        Y = torch.empty((M, down.N), dtype=out_dtype or X.dtype, device=dev)
    if save_z and Z_up is None:
        Z_up = torch.empty((M, up.N), dtype=X.dtype, device=dev)
    _need(H, "H", (M, up.N), (X.dtype,), dev)
    _need(Y, "Y", (M, down.N), _FLOATS, dev)
    if save_z:
        _need(Z_up, "Z_up", (M, up.N), (X.dtype,), dev)
    _gpu(dev)
    ws, nbytes = _ws("ffn_fwd", up, down, M, dev, ws)
    _check(LIB.star_ffn_fwd(up.ref, down.ref, M, _ptr(row_type), _ptr(X), _ptr(W_up), _ptr(b_up),
                            _ptr(W_down), _ptr(b_down), ACTS[act], _ptr(Z_up) if save_z else None,
                            _ptr(H), _ptr(Y), _dt(X), _dt(Y), _ptr(ws), nbytes, _stream(dev)),
           "star_ffn_fwd")
    return (Z_up if save_z else None), H, Y


def _decode_args(up: Algebra, down: Algebra, row_type, X, L: int, Y, out_dtype, weights, biases):
    if not isinstance(X, torch.Tensor) or X.dtype != torch.bfloat16:
        raise TypeError("decode takes a bfloat16 X")
    M, dev = _rows(X, "X", up.K)
    _types(row_type, M, dev)
    if down.K != up.N or down.N != up.K:
        raise ValueError("down must map the up projection's output back to its input width")
    for name, ts, shape in weights:
        if len(ts) != L:
            raise ValueError(f"{name} needs one tensor per layer ({L})")
        for t in ts:
            _need(t, name, shape, _BF16, dev)
    for name, ts, shape in biases:
        if ts is None:
            continue
        if len(ts) != L:
            raise ValueError(f"{name} needs one entry per layer ({L})")
        for t in ts:
            _opt(t, name, shape, _F32, dev)
    if Y is None:
        Y = torch.empty((M, up.K), dtype=out_dtype or X.dtype, device=dev)
    _need(Y, "Y", (M, up.K), _FLOATS, dev)
    return M, dev, Y


def star_decode_status(ws: torch.Tensor) -> bool:
    """True when the last decode call on workspace ``ws`` lost its step to a
    wait bound (its Y is then unspecified).  Synchronises the stream."""
    flag = ctypes.c_int32()
    _need(ws, "ws", tuple(ws.shape))
    _gpu(ws.device)
    _check(LIB.star_decode_status(_ptr(ws), ws.numel() * ws.element_size(), ctypes.byref(flag),
                                  _stream(ws.device)), "star_decode_status")
    return bool(flag.value)


def _decode_checked(ws, check: bool, where: str):
    if check and star_decode_status(ws):
        raise RuntimeError(f"{where}: a wait of the decode stack ran out (the device was not free "
                           "for all of its workgroups); the step's output is unspecified")


def star_decode(up: Algebra, down: Algebra, row_type: torch.Tensor, X: torch.Tensor,
                W_ups: Sequence[torch.Tensor], b_ups, W_downs: Sequence[torch.Tensor], b_downs,
                act: str = "gelu", residual: bool = True, Y=None, out_dtype=None, ws=None,
                check: bool = True):
    """One decode step through ``len(W_ups)`` FFN layers; returns Y.  With
    ``check`` (the default) the call synchronises and raises if the step was
    lost to a wait bound; pass ``check=False`` (and a ``ws`` to read with
    ``star_decode_status`` later) inside timed loops and graph captures."""
    L = len(W_ups)
    M, dev, Y = _decode_args(up, down, row_type, X, L, Y, out_dtype,
                             [("W_up", W_ups, (up.K, up.N)), ("W_down", W_downs, (down.K, down.N))],
                             [("b_up", b_ups, (up.N,)), ("b_down", b_downs, (down.N,))])
    P = ctypes.c_void_p
    wu = (P * L)(*[t.data_ptr() for t in W_ups])
    wd = (P * L)(*[t.data_ptr() for t in W_downs])
    bu = (P * L)(*[t.data_ptr() if t is not None else None for t in b_ups]) if b_ups is not None else None
    bd = (P * L)(*[t.data_ptr() if t is not None else None for t in b_downs]) if b_downs is not None else None
    _gpu(dev)
    ws, nbytes = _ws("decode", up, down, M, dev, ws)
    _check(LIB.star_decode(up.ref, down.ref, L, M, _ptr(row_type), _ptr(X), _dt(X), wu, bu, wd, bd,
                           ACTS[act], int(bool(residual)), _ptr(Y), _dt(Y), _ptr(ws), nbytes,
                           _stream(dev)), "star_decode")
    _decode_checked(ws, check, "star_decode")
    return Y


def star_decode_noalloc(up: Algebra, down: Algebra, row_type: torch.Tensor, X: torch.Tensor,
                        W_ups: Sequence[torch.Tensor], b_ups, W_downs: Sequence[torch.Tensor], b_downs,
                        act: str = "gelu", residual: bool = True, Y=None, out_dtype=None, status=None):
    """star_decode on the library's static workspace (the C entry point
    allocates nothing; this wrapper allocates Y only when none is given).
    ``status``: a device int32 tensor of one element (or None) that receives
    the step's wait-bound flag.  Returns Y."""
    L = len(W_ups)
    M, dev, Y = _decode_args(up, down, row_type, X, L, Y, out_dtype,
                             [("W_up", W_ups, (up.K, up.N)), ("W_down", W_downs, (down.K, down.N))],
                             [("b_up", b_ups, (up.N,)), ("b_down", b_downs, (down.N,))])
    _opt(status, "status", (1,), _I32, dev)
    P = ctypes.c_void_p
    wu = (P * L)(*[t.data_ptr() for t in W_ups])
    wd = (P * L)(*[t.data_ptr() for t in W_downs])
    bu = (P * L)(*[t.data_ptr() if t is not None else None for t in b_ups]) if b_ups is not None else None
    bd = (P * L)(*[t.data_ptr() if t is not None else None for t in b_downs]) if b_downs is not None else None
    _gpu(dev)
    _check(LIB.star_decode_noalloc(up.ref, down.ref, L, M, _ptr(row_type), _ptr(X), _dt(X), wu, bu, wd, bd,
                                   ACTS[act], int(bool(residual)), _ptr(Y), _dt(Y), _ptr(status),
                                   _stream(dev)), "star_decode_noalloc")
    return Y


def star_decode_gated(up: Algebra, down: Algebra, row_type: torch.Tensor, X: torch.Tensor,
                      W_gates: Sequence[torch.Tensor], b_gates, W_ups: Sequence[torch.Tensor], b_ups,
                      W_downs: Sequence[torch.Tensor], b_downs, residual: bool = True, Y=None,
                      out_dtype=None, ws=None, check: bool = True):
    """One decode step through ``len(W_ups)`` gated-FFN (SwiGLU) layers;
    returns Y (``check`` as in star_decode)."""
    L = len(W_ups)
    M, dev, Y = _decode_args(up, down, row_type, X, L, Y, out_dtype,
                             [("W_gate", W_gates, (up.K, up.N)), ("W_up", W_ups, (up.K, up.N)),
                              ("W_down", W_downs, (down.K, down.N))],
                             [("b_gate", b_gates, (up.N,)), ("b_up", b_ups, (up.N,)),
                              ("b_down", b_downs, (down.N,))])
    P = ctypes.c_void_p
    arr = lambda ts: (P * L)(*[t.data_ptr() for t in ts])
    opt = lambda ts: (P * L)(*[t.data_ptr() if t is not None else None for t in ts]) if ts is not None else None
    _gpu(dev)
    ws, nbytes = _ws("decode", up, down, M, dev, ws)
    _check(LIB.star_decode_gated(up.ref, down.ref, L, M, _ptr(row_type), _ptr(X), _dt(X), arr(W_gates),
                                 opt(b_gates), arr(W_ups), opt(b_ups), arr(W_downs), opt(b_downs),
                                 int(bool(residual)), _ptr(Y), _dt(Y), _ptr(ws), nbytes, _stream(dev)),
           "star_decode_gated")
    _decode_checked(ws, check, "star_decode_gated")
    return Y


def star_ffn_bwd(up: Algebra, down: Algebra, row_type: torch.Tensor, X: torch.Tensor,
                 Z_up: torch.Tensor, H: torch.Tensor, W_up: torch.Tensor, W_down: torch.Tensor,
                 dY: torch.Tensor, act: str = "gelu", plan=None, ws=None):
    """Backward of ``star_ffn_fwd``: one type plan, then four library calls
    on one stream: dZ = (dY *^T W_down) . act'(Z_up) (fused epilogue);
    dW_down, db_down from (H, dY); dW_up, db_up from (X, dZ); dX = dZ *^T W_up.
    Returns a dict of dX, dZ, dW_up, db_up, dW_down, db_down."""
    if plan is None:
        plan = star_type_plan(up.q, row_type)
    dZ = star_proj_bwd_data_planned(down, plan, dY, W_down, Z_prev=Z_up, act_prev=act,
                                    out_dtype=X.dtype)
    dW_down, db_down = star_proj_bwd_weight_planned(down, plan, H, dY, ws=ws)
    dW_up, db_up = star_proj_bwd_weight_planned(up, plan, X, dZ, ws=ws)
    dX = star_proj_bwd_data_planned(up, plan, dZ, W_up)
    return dict(dX=dX, dZ=dZ, dW_up=dW_up, db_up=db_up, dW_down=dW_down, db_down=db_down)


# ---- gated FFN (SwiGLU) --------------------------------------------------------------


def star_swiglu_fwd(Z_gate: torch.Tensor, Z_up: torch.Tensor, H=None) -> torch.Tensor:
    """H = silu(Z_gate) . Z_up (elementwise, on the GPU)."""
    _need(Z_gate, "Z_gate", tuple(Z_gate.shape), _FLOATS)
    _need(Z_up, "Z_up", tuple(Z_gate.shape), (Z_gate.dtype,), Z_gate.device)
    if H is None:
        H = torch.empty_like(Z_gate)
    _need(H, "H", tuple(Z_gate.shape), (Z_gate.dtype,), Z_gate.device)
    _gpu(Z_gate.device)
    _check(LIB.star_swiglu_fwd(Z_gate.numel(), _ptr(Z_gate), _ptr(Z_up), _dt(Z_gate), _ptr(H),
                               _stream(Z_gate.device)), "star_swiglu_fwd")
    return H


def pack_gate_up(gate: torch.Tensor, up: torch.Tensor) -> torch.Tensor:
    """The merged gate/up layout of star_swiglu_up_fwd_planned: the last
    dimension (F, a multiple of 8) of ``gate`` and ``up`` interleaved in
    8-wide chunks (gate chunk c, then up chunk c).  A one-time layout
    conversion of the weights W [D, F] or biases [F] (torch ops; not part of
    the product)."""
    if gate.shape != up.shape or gate.shape[-1] % 8:
        raise ValueError("gate and up need the same shape, the last dimension a multiple of 8")
    lead, F = tuple(gate.shape[:-1]), gate.shape[-1]
    g = gate.reshape(*lead, F // 8, 1, 8)
    u = up.reshape(*lead, F // 8, 1, 8)
    return torch.cat((g, u), dim=-2).reshape(*lead, 2 * F).contiguous()


def star_swiglu_merged_fwd(Z_gu: torch.Tensor, H=None) -> torch.Tensor:
    """H [M, F] = silu(gate) . up from a merged gate/up output Z_gu [M, 2F]
    (gate and up interleaved in 8-feature chunks; elementwise, on the GPU)."""
    if Z_gu.dim() != 2 or Z_gu.shape[1] % 16:
        raise ValueError("Z_gu must be [M, 2F] with F a multiple of 8")
    M, F = Z_gu.shape[0], Z_gu.shape[1] // 2
    _need(Z_gu, "Z_gu", (M, 2 * F), _FLOATS)
    if H is None:
        H = torch.empty((M, F), dtype=Z_gu.dtype, device=Z_gu.device)
    _need(H, "H", (M, F), (Z_gu.dtype,), Z_gu.device)
    _gpu(Z_gu.device)
    _check(LIB.star_swiglu_merged_fwd(M, F, _ptr(Z_gu), _dt(Z_gu), _ptr(H), _stream(Z_gu.device)),
           "star_swiglu_merged_fwd")
    return H


def star_swiglu_up_fwd_planned(alg_gu: Algebra, plan: torch.Tensor, X: torch.Tensor, W_gu: torch.Tensor,
                               b_gu: torch.Tensor | None = None, Z_out=None, H=None, out_dtype=None):
    """H = silu(Z_gate) . Z_up of the merged gate/up product X *_q W_gu
    (+ b_gu), SwiGLU applied in the product's epilogue.  ``alg_gu`` is the
    merged algebra (Algebra.merged_gate_up), W_gu and b_gu from pack_gate_up.
    ``Z_out=True`` also returns the merged pre-activation [M, 2F].  Returns H,
    or (H, Z)."""
    M, dev = _rows(X, "X", alg_gu.K)
    _need(W_gu, "W_gu", (alg_gu.K, alg_gu.N), (X.dtype,), dev)
    _opt(b_gu, "b_gu", (alg_gu.N,), _F32, dev)
    _need(plan, "plan", tuple(plan.shape), None, dev)
    F = alg_gu.N // 2
    if H is None:
        H = torch.empty((M, F), dtype=out_dtype or X.dtype, device=dev)
    _need(H, "H", (M, F), _FLOATS, dev)
    want_z = Z_out is not None and Z_out is not False
    if Z_out is True:
        Z_out = torch.empty((M, alg_gu.N), dtype=H.dtype, device=dev)
    if want_z:
        _need(Z_out, "Z_out", (M, alg_gu.N), (H.dtype,), dev)
    _gpu(dev)
    _check(LIB.star_swiglu_up_fwd_planned(alg_gu.ref, M, _ptr(plan), _ptr(X), _dt(X), _ptr(W_gu), _dt(W_gu),
                                          _ptr(b_gu), _ptr(Z_out) if want_z else None, _ptr(H), _dt(H),
                                          _stream(dev)), "star_swiglu_up_fwd_planned")
    return (H, Z_out) if want_z else H


def star_swiglu_bwd(dH: torch.Tensor, Z_gate: torch.Tensor, Z_up: torch.Tensor):
    """(dZ_gate, dZ_up) = (dH . Z_up . silu'(Z_gate), dH . silu(Z_gate))."""
    _need(dH, "dH", tuple(dH.shape), _FLOATS)
    _need(Z_gate, "Z_gate", tuple(dH.shape), (dH.dtype,), dH.device)
    _need(Z_up, "Z_up", tuple(dH.shape), (dH.dtype,), dH.device)
    dZg, dZu = torch.empty_like(dH), torch.empty_like(dH)
    _gpu(dH.device)
    _check(LIB.star_swiglu_bwd(dH.numel(), _ptr(dH), _ptr(Z_gate), _ptr(Z_up), _dt(dH), _ptr(dZg),
                               _ptr(dZu), _stream(dH.device)), "star_swiglu_bwd")
    return dZg, dZu


def star_add(a: torch.Tensor, b: torch.Tensor, out=None) -> torch.Tensor:
    """out = a + b (elementwise, on the GPU; out may be a or b)."""
    _need(a, "a", tuple(a.shape), _FLOATS)
    _need(b, "b", tuple(a.shape), (a.dtype,), a.device)
    if out is None:
        out = torch.empty_like(a)
    _need(out, "out", tuple(a.shape), (a.dtype,), a.device)
    _gpu(a.device)
    _check(LIB.star_add(a.numel(), _ptr(a), _ptr(b), _dt(a), _ptr(out), _stream(a.device)), "star_add")
    return out


def star_swiglu_ffn_fwd(up: Algebra, down: Algebra, row_type: torch.Tensor, X: torch.Tensor,
                        W_gate: torch.Tensor, b_gate, W_up: torch.Tensor, b_up, W_down: torch.Tensor,
                        b_down, plan=None, out_dtype=None):
    """Gated FFN with one type plan for its three projections:
    Z_g = X *_q W_gate + b_gate, Z_u = X *_q W_up + b_up, H = silu(Z_g) . Z_u,
    Y = H *_q W_down + b_down.  Returns (Z_g, Z_u, H, Y)."""
    if plan is None:
        plan = star_type_plan(up.q, row_type)
    Zg = star_proj_fwd_planned(up, plan, X, W_gate, b_gate, "none")
    Zu = star_proj_fwd_planned(up, plan, X, W_up, b_up, "none")
    H = star_swiglu_fwd(Zg, Zu)
    Y = star_proj_fwd_planned(down, plan, H, W_down, b_down, "none", out_dtype=out_dtype)
    return Zg, Zu, H, Y


def star_swiglu_ffn_bwd(up: Algebra, down: Algebra, row_type: torch.Tensor, X: torch.Tensor,
                        Z_gate: torch.Tensor, Z_up: torch.Tensor, H: torch.Tensor, W_gate: torch.Tensor,
                        W_up: torch.Tensor, W_down: torch.Tensor, dY: torch.Tensor, plan=None, ws=None):
    """Backward of ``star_swiglu_ffn_fwd``: dH = dY *^T W_down; the gate's
    elementwise backward; dX = dZ_g *^T W_gate + dZ_u *^T W_up; the three
    weight and bias gradients.  Returns a dict of dX, dZ_gate, dZ_up,
    dW_gate, db_gate, dW_up, db_up, dW_down, db_down."""
    if plan is None:
        plan = star_type_plan(up.q, row_type)
    dH = star_proj_bwd_data_planned(down, plan, dY, W_down, out_dtype=X.dtype)
    dZg, dZu = star_swiglu_bwd(dH, Z_gate, Z_up)
    dW_down, db_down = star_proj_bwd_weight_planned(down, plan, H, dY, ws=ws)
    dW_gate, db_gate = star_proj_bwd_weight_planned(up, plan, X, dZg, ws=ws)
    dW_up, db_up = star_proj_bwd_weight_planned(up, plan, X, dZu, ws=ws)
    # the two input gradients in fp32, summed once
    dX = star_proj_bwd_data_planned(up, plan, dZg, W_gate, out_dtype=torch.float32)
    dX = star_add(dX, star_proj_bwd_data_planned(up, plan, dZu, W_up, out_dtype=torch.float32), out=dX)
    return dict(dX=dX, dZ_gate=dZg, dZ_up=dZu, dW_gate=dW_gate, db_gate=db_gate, dW_up=dW_up,
                db_up=db_up, dW_down=dW_down, db_down=db_down)


# ---- algebraic attention ------------------------------------------------------

class AttnShape:
    """Shape of an algebraic-attention call: ``batch`` sequences of
    ``seq_len`` positions (the cache capacity for decode), ``n_heads`` query
    and ``n_kv_heads`` key/value heads of width ``head_dim`` = q m, under
    ``law`` ("star", "dense" or "tensor2")."""

    def __init__(self, batch: int, seq_len: int, n_heads: int, n_kv_heads: int, head_dim: int, q: int,
                 law: str = "star"):
        self.batch, self.seq_len, self.n_heads = int(batch), int(seq_len), int(n_heads)
        self.n_kv_heads, self.head_dim, self.q, self.law = int(n_kv_heads), int(head_dim), int(q), law
        self._c = _CAttnShape(self.batch, self.seq_len, self.n_heads, self.n_kv_heads, self.head_dim,
                              self.q, LAWS[law])

    @property
    def ref(self):
        return ctypes.byref(self._c)

    def with_law(self, law: str) -> "AttnShape":
        return AttnShape(self.batch, self.seq_len, self.n_heads, self.n_kv_heads, self.head_dim, self.q, law)

    def __repr__(self):
        return (f"AttnShape(batch={self.batch}, seq_len={self.seq_len}, n_heads={self.n_heads}, "
                f"n_kv_heads={self.n_kv_heads}, head_dim={self.head_dim}, q={self.q}, law={self.law!r})")


def star_attn_fwd(shape: AttnShape, plan: torch.Tensor, Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor,
                  O=None, out_dtype=torch.bfloat16, lse=None, want_lse: bool = False):
    """Causal algebraic attention over whole sequences.  ``plan`` is the type
    plan of the position types (``star_type_plan(q, pos_type)``); Q is
    [B, S, n_heads, d_h], K and V [B, S, n_kv_heads, d_h], bf16.  Returns O
    (and the log-sum-exp [B, n_heads, S] when ``want_lse`` or ``lse`` is
    given)."""
    B, S, H, Hkv, D = shape.batch, shape.seq_len, shape.n_heads, shape.n_kv_heads, shape.head_dim
    dev = Q.device if isinstance(Q, torch.Tensor) else None
    _need(Q, "Q", (B, S, H, D), _BF16, dev)
    _need(K, "K", (B, S, Hkv, D), _BF16, dev)
    _need(V, "V", (B, S, Hkv, D), _BF16, dev)
    _need(plan, "plan", tuple(plan.shape), None, dev)
    if O is None:
        O = torch.empty((B, S, H, D), dtype=out_dtype, device=dev)
    _need(O, "O", (B, S, H, D), _FLOATS, dev)
    if lse is None and want_lse:
        lse = torch.empty((B, H, S), dtype=torch.float32, device=dev)
    _opt(lse, "lse", (B, H, S), _F32, dev)
    _gpu(dev)
    _check(LIB.star_attn_fwd(shape.ref, _ptr(plan), _ptr(Q), _ptr(K), _ptr(V), DTYPES[torch.bfloat16], _ptr(O),
                             _dt(O), _ptr(lse), _stream(dev)), "star_attn_fwd")
    return (O, lse) if lse is not None else O


def star_attn_decode_workspace_bytes(shape: AttnShape) -> int:
    return int(LIB.star_attn_decode_workspace_bytes(shape.ref))


def star_attn_decode(shape: AttnShape, pos_type: torch.Tensor, cache_len: torch.Tensor, Q: torch.Tensor,
                     K_cache: torch.Tensor, V_cache: torch.Tensor, O=None, out_dtype=torch.bfloat16, ws=None):
    """One decode step: Q [B, n_heads, d_h] against the caches
    [B, S_max, n_kv_heads, d_h] (bf16), ``cache_len`` [B] valid entries per
    sequence (the query sits at position cache_len - 1), ``pos_type``
    [S_max].  Returns O [B, n_heads, d_h]."""
    B, S, H, Hkv, D = shape.batch, shape.seq_len, shape.n_heads, shape.n_kv_heads, shape.head_dim
    dev = Q.device if isinstance(Q, torch.Tensor) else None
    _need(Q, "Q", (B, H, D), _BF16, dev)
    _need(K_cache, "K_cache", (B, S, Hkv, D), _BF16, dev)
    _need(V_cache, "V_cache", (B, S, Hkv, D), _BF16, dev)
    _need(pos_type, "pos_type", (S,), _I32, dev)
    _need(cache_len, "cache_len", (B,), _I32, dev)
    if O is None:
        O = torch.empty((B, H, D), dtype=out_dtype, device=dev)
    _need(O, "O", (B, H, D), _FLOATS, dev)
    need = star_attn_decode_workspace_bytes(shape)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    _need(ws, "ws", tuple(ws.shape), None, dev)
    _gpu(dev)
    _check(LIB.star_attn_decode(shape.ref, _ptr(pos_type), _ptr(cache_len), _ptr(Q), _ptr(K_cache),
                                _ptr(V_cache), DTYPES[torch.bfloat16], _ptr(O), _dt(O), _ptr(ws),
                                ws.numel() * ws.element_size(), _stream(dev)), "star_attn_decode")
    return O
