"""Host-only checks of the C ABI: the library loads, exports every entry point
the header declares, and rejects bad arguments before launching anything.
No test here launches a kernel, so all run without a GPU."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "star_proj.h")


@pytest.fixture(scope="module")
def P():
    import paper_2609_32814_amd as P
    return P


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(star_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(P):
    names = declared_functions()
    assert {"star_proj_fwd", "star_proj_bwd_data", "star_proj_bwd_weight", "star_ffn_fwd",
            "star_decode"} <= set(names)
    lib = ctypes.CDLL(P.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_binding_names_match_abi(P):
    for n in declared_functions():
        assert hasattr(P, n), n


def test_set_fwd_tiles(P):
    assert P.star_set_fwd_tiles("wide") == "auto"
    assert P.star_set_fwd_tiles("small") == "wide"
    assert P.star_set_fwd_tiles("wide192") == "small"
    assert P.star_set_fwd_tiles("auto") == "wide192"
    with pytest.raises(ValueError):
        P.star_set_fwd_tiles("huge")
    lib = ctypes.CDLL(P.LIB_PATH)
    lib.star_set_fwd_tiles.restype = ctypes.c_int
    assert lib.star_set_fwd_tiles(4) == -1 and lib.star_set_fwd_tiles(-1) == -1
    assert P.star_set_fwd_tiles("auto") == "auto"


def test_pack_gate_up_layout(P):
    """Gate and up interleaved in 8-wide chunks of the last axis (CPU)."""
    import torch
    g = torch.arange(3 * 96, dtype=torch.float32).reshape(3, 96)
    u = -g - 1
    m = P.pack_gate_up(g, u)
    assert m.shape == (3, 192)
    for c in range(12):
        assert torch.equal(m[:, 16 * c:16 * c + 8], g[:, 8 * c:8 * c + 8])
        assert torch.equal(m[:, 16 * c + 8:16 * c + 16], u[:, 8 * c:8 * c + 8])
    assert torch.equal(P.pack_gate_up(g[0], u[0]), m[0])
    with pytest.raises(ValueError):
        P.pack_gate_up(g[:, :44], u[:, :44])


def test_swiglu_merged_argument_errors(P):
    """The merged gate/up calls refuse what they do not take, on the host."""
    import numpy as np
    import paper_2609_32814_amd.binding as B
    err = {v: k for k, v in P.binding.STATUS_NAMES.items()}
    V = ctypes.c_void_p
    L = P.binding.LIB

    def fused(alg, xt=1, ht=1):
        return L.star_swiglu_up_fwd_planned(alg.ref, 4, V(16), V(16), xt, V(16), xt, None, None, V(16), ht, None)

    good = B.Algebra.equal(2, 64, 128).merged_gate_up()
    assert fused(B.Algebra(2, [64, 64], [88, 64])) == err["STAR_ERR_UNSUPPORTED"]  # merged width not 16k
    assert fused(good, xt=0) == err["STAR_ERR_UNSUPPORTED"]                        # fp32 operands
    E = np.array([[0, 1], [0, 0]], np.uint8)
    assert fused(B.Algebra(2, [64, 64], [128, 128], "graph", E)) == err["STAR_ERR_UNSUPPORTED"]
    assert L.star_swiglu_merged_fwd(4, 44, V(16), 1, V(16), None) == err["STAR_ERR_ALIGN"]  # F not 8k
    assert L.star_swiglu_merged_fwd(4, 64, V(16), 7, V(16), None) == err["STAR_ERR_DTYPE"]
    assert L.star_swiglu_merged_fwd(4, 64, None, 1, V(16), None) == err["STAR_ERR_ARG"]
    assert L.star_swiglu_merged_fwd(0, 64, None, 1, None, None) == 0                       # M = 0: no-op


def test_count_products(P):
    for q in (1, 2, 3, 8, 16, 64):
        a = P.Algebra.equal(q, 8 * q, 8 * q)
        assert P.star_count_products(a) == [2 * q - 1] * q
        assert P.star_count_products(a.with_law("dense")) == [q * q] * q


def test_count_macs_closed_form(P):
    """eq. rectangular-batch-cost: M D_diag + sum_i M_i s_i (N - r_i)."""
    s, r = [8, 40, 16], [24, 8, 56]
    a = P.Algebra(3, s, r)
    rows = [5, 0, 11]
    D = sum(x * y for x, y in zip(s, r))
    N = sum(r)
    expect = sum(rows) * D + sum(m * si * (N - ri) for m, si, ri in zip(rows, s, r))
    assert P.star_count_macs(a, rows) == expect
    assert P.star_count_macs(a.with_law("dense"), rows) == sum(rows) * sum(s) * N


def test_workspace_sizes(P):
    a = P.Algebra.equal(2, 768, 3072)
    d = P.Algebra.equal(2, 3072, 768)
    fwd = P.star_workspace_bytes("fwd", a, None, 8192)
    assert fwd >= 4 * 8192 + 4 * 3
    bw = P.star_workspace_bytes("bwd_weight", a, None, 16384)
    assert bw >= fwd
    dec = P.star_workspace_bytes("decode", a, d, 64)
    assert dec >= 64 * 768 * 4 + 64 * 768 * 2 + 64 * 3072 * 2
    assert P.star_workspace_bytes("fwd", P.Algebra(2, [7, 9], [8, 8]), None, 10) == 0
    # projections wider than 4096 decode one launch per projection
    wu, wd = P.Algebra.equal(4, 1024, 8192), P.Algebra.equal(4, 8192, 1024)
    assert P.star_workspace_bytes("decode", wu, wd, 16) >= 16 * 1024 * 4 + 16 * 8192 * 2


def _raw_fwd(P, alg_c, M, xt=1, wt=1, yt=1, X=16, W=16, Y=16, ws=16, ws_bytes=1 << 20,
             rt=16, act=0):
    # fake, aligned, never-dereferenced pointers: these calls must fail validation
    V = ctypes.c_void_p
    return P.binding.LIB.star_proj_fwd(alg_c, M, V(rt) if rt else None, V(X) if X else None, xt,
                                       V(W) if W else None, wt, None, act, None,
                                       V(Y) if Y else None, yt, V(ws) if ws else None, ws_bytes,
                                       None)


def test_argument_errors_before_launch(P):
    import paper_2609_32814_amd.binding as B
    good = P.Algebra.equal(2, 64, 64)
    assert _raw_fwd(P, None, 4) == 1                                   # null algebra
    assert _raw_fwd(P, P.Algebra(2, [12, 52], [32, 32]).ref, 4) == 4   # width not multiple of 8
    assert _raw_fwd(P, good.ref, 4, xt=0, wt=1) == 3                   # mixed operand dtypes
    assert _raw_fwd(P, good.ref, 4, yt=5) == 3                         # bad dtype
    assert _raw_fwd(P, good.ref, 4, act=9) == 1                        # bad activation
    assert _raw_fwd(P, good.ref, 4, X=0) == 1                          # null operand
    assert _raw_fwd(P, good.ref, 4, X=18) == 4                         # misaligned operand
    assert _raw_fwd(P, good.ref, 4, ws_bytes=8) == 5                   # workspace too small
    assert _raw_fwd(P, good.ref, 4, ws=0) == 5                         # no workspace
    assert _raw_fwd(P, good.ref, -1) == 2                              # negative M
    assert _raw_fwd(P, good.ref, 0, X=0, W=0, Y=0, ws=0, rt=0) == 0    # M = 0: no-op
    big = B.Algebra(257, [8] * 257, [8] * 257)
    assert _raw_fwd(P, big.ref, 4) == 1                                # q above STAR_MAX_Q_FWD
    assert P.star_status_string(5).startswith("workspace")


def test_large_q_limits(P):
    """q in (64, 256]: the forward product of the star and dense laws with
    bf16 operands, the plan and the counting helpers take it; everything
    else refuses it on the host (fake pointers, nothing launched)."""
    import numpy as np
    import paper_2609_32814_amd.binding as B
    err = {v: k for k, v in P.binding.STATUS_NAMES.items()}
    a128 = B.Algebra.equal(128, 16 * 128, 40 * 128)
    assert P.star_count_products(a128) == [255] * 128
    assert P.star_count_products(B.Algebra.equal(256, 8 * 256, 8 * 256)) == [511] * 256
    assert P.star_count_macs(a128, [1] * 128) == 128 * 40 * 16 * (1 + 2 * 127)
    assert P.star_workspace_bytes("fwd", a128, None, 1000) >= 4 * 1000 + 4 * 129
    assert P.star_workspace_bytes("bwd_data", a128, None, 1000) == 0
    assert P.star_workspace_bytes("bwd_weight", a128, None, 1000) == 0
    assert P.star_plan_bytes(256, 10) > 0 and P.star_plan_bytes(257, 10) == 0
    assert _raw_fwd(P, a128.ref, 4, xt=0, wt=0, yt=0) == err["STAR_ERR_UNSUPPORTED"]  # fp32 operands
    E = np.zeros((65, 65), np.uint8)
    E[0, 1] = 1
    g65 = B.Algebra(65, [8] * 65, [8] * 65, "graph", E)
    assert _raw_fwd(P, g65.ref, 4) == err["STAR_ERR_UNSUPPORTED"]                      # graph law
    V = ctypes.c_void_p
    st = P.binding.LIB.star_proj_bwd_data(a128.ref, 4, V(16), V(16), 1, V(16), 1, None, 0, V(16), 1,
                                          V(16), 1 << 20, None)
    assert st == err["STAR_ERR_UNSUPPORTED"]
    assert P.binding.LIB.star_type_plan(257, 4, V(16), V(16), 1 << 20, None) == err["STAR_ERR_ARG"]


def test_decode_rejects_too_many_rows(P):
    V = ctypes.c_void_p
    up, dn = P.Algebra.equal(2, 64, 128), P.Algebra.equal(2, 128, 64)
    arr = (V * 1)(V(16))
    st = P.binding.LIB.star_decode(up.ref, dn.ref, 1, 65, V(16), V(16), 1, arr, None, arr, None, 1,
                                   1, V(16), 1, V(16), 1 << 30, None)
    assert st == 6
    st = P.binding.LIB.star_decode(up.ref, P.Algebra.equal(2, 128, 32).ref, 1, 4, V(16), V(16), 1,
                                   arr, None, arr, None, 1, 1, V(16), 1, V(16), 1 << 30, None)
    assert st == 2
    # X must be bfloat16
    st = P.binding.LIB.star_decode(up.ref, dn.ref, 1, 4, V(16), V(16), 0, arr, None, arr, None, 1,
                                   1, V(16), 1, V(16), 1 << 30, None)
    assert st == 3


def test_decode_status_argument_errors(P):
    """The status call checks its arguments on the host (no device access)."""
    V = ctypes.c_void_p
    flag = ctypes.c_int32(7)
    assert P.binding.LIB.star_decode_status(None, 16, ctypes.byref(flag), None) == 1
    assert P.binding.LIB.star_decode_status(V(16), 16, None, None) == 1
    assert P.binding.LIB.star_decode_status(V(16), 2, ctypes.byref(flag), None) == 5
    assert P.binding.LIB.star_decode_status(V(8), 16, ctypes.byref(flag), None) == 4
    assert flag.value == 7


def test_binding_refuses_bad_tensors(P):
    """The binding checks shapes, dtypes, contiguity and devices before any
    pointer crosses the ABI (CPU tensors are refused too, so this runs here)."""
    import torch
    alg = P.Algebra.equal(2, 64, 128)
    X = torch.zeros(8, 64)
    W = torch.zeros(64, 128)
    t = torch.zeros(8, dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU tensor"):
        P.star_proj_fwd(alg, t, X, W)
    with pytest.raises(ValueError, match="shape"):
        P.star_proj_fwd(alg, t, torch.zeros(8, 65), W)
    with pytest.raises(ValueError, match="shape"):
        P.star_proj_fwd(alg, t, X, torch.zeros(64, 127))
    with pytest.raises(TypeError, match="dtype"):
        P.star_proj_fwd(alg, t, X, W.to(torch.bfloat16))
    with pytest.raises(TypeError, match="dtype"):
        P.star_proj_fwd(alg, t.to(torch.int64), X, W)
    with pytest.raises(ValueError, match="shape"):
        P.star_proj_fwd(alg, t[:7], X, W)
    with pytest.raises(ValueError, match="contiguous"):
        P.star_proj_fwd(alg, t, torch.zeros(64, 8).t(), W)
    with pytest.raises(ValueError, match="shape"):
        P.star_proj_bwd_weight(alg, t, X, torch.zeros(8, 64))
    up, dn = P.Algebra.equal(2, 64, 128), P.Algebra.equal(2, 128, 64)
    with pytest.raises(TypeError, match="bfloat16"):
        P.star_decode(up, dn, t, X, [W.to(torch.bfloat16)], None, [W.t().contiguous().to(torch.bfloat16)], None)


def test_ffn_rejects_mismatched_widths(P):
    V = ctypes.c_void_p
    up, dn = P.Algebra(2, [32, 32], [64, 64]), P.Algebra(2, [56, 72], [32, 32])
    st = P.binding.LIB.star_ffn_fwd(up.ref, dn.ref, 4, V(16), V(16), V(16), None, V(16), None, 1,
                                    None, V(16), V(16), 1, 1, V(16), 1 << 20, None)
    assert st == 2


def test_tensor_power_law_counts_and_limits(P):
    """Law TENSOR2: 9 block products per type at q = 4 (36 in all, the
    paper's count), the two-group law at q = 2, MACs against the oracle's
    support, and q outside {1, 2, 4} refused before any launch."""
    import oracle
    a = P.Algebra.equal(4, 768, 3072, "tensor2")
    assert P.star_count_products(a) == [9] * 4
    assert P.star_count_products(P.Algebra.equal(2, 64, 64, "tensor2")) == [3, 3]
    rows = [5, 0, 7, 3]
    oa = oracle.Alg.equal(4, 768, 3072, "tensor2")
    assert P.star_count_macs(a, rows) == sum(n * oracle.row_macs(oa, i) for i, n in enumerate(rows))
    with pytest.raises(RuntimeError):
        P.star_count_products(P.Algebra.equal(8, 64, 64, "tensor2"))


def test_graph_law_counts_and_arguments(P):
    """Law "graph": per-type products 1 + 2 outdeg(i) (eq. graph-rank: |V| +
    2|E| over all types), MACs from the same support, and the ABI refuses the
    law without an edge matrix."""
    import numpy as np
    import oracle
    E = np.array([[0, 1, 1, 0], [0, 0, 0, 1], [1, 0, 0, 0], [0, 0, 0, 0]], np.uint8)
    a = P.Algebra(4, [8, 16, 24, 8], [16, 8, 8, 32], "graph", E)
    per = P.star_count_products(a)
    assert per == [1 + 2 * int(E[i].sum()) for i in range(4)]
    assert sum(per) == 4 + 2 * int(E.sum())
    oa = oracle.Alg(4, a.s, a.r, "graph", tuple(map(tuple, E)))
    rows = [5, 0, 7, 3]
    assert P.star_count_macs(a, rows) == sum(n * oracle.row_macs(oa, i) for i, n in enumerate(rows))
    # the diagonal of the edge matrix is ignored
    E2 = E.copy()
    np.fill_diagonal(E2, 1)
    assert P.star_count_products(P.Algebra(4, a.s, a.r, "graph", E2)) == per
    # no edge matrix: STAR_ERR_ARG from the ABI itself
    bare = P.binding._CAlgebra(a._c.q, a._c.s, a._c.r, 3, None)
    out = (ctypes.c_int64 * 4)()
    assert P.binding.LIB.star_count_products(ctypes.byref(bare), out) == 1
    with pytest.raises(ValueError):
        P.Algebra(2, [8, 8], [8, 8], "graph")


def _attn_shape(P, **kw):
    base = dict(batch=2, seq_len=100, n_heads=4, n_kv_heads=2, head_dim=64, q=4, law=0)
    base.update(kw)
    return P.binding._CAttnShape(**base)


def _raw_attn_fwd(P, sh, dt=1, ot=0, ptrs=16, lse=None):
    V = ctypes.c_void_p
    p = V(ptrs) if ptrs else None
    return P.binding.LIB.star_attn_fwd(ctypes.byref(sh), p, p, p, p, dt, p, ot, V(lse) if lse else None, None)


def _raw_attn_dec(P, sh, ws_bytes=1 << 20, ptr=16, ws=16):
    V = ctypes.c_void_p
    p = V(ptr)
    return P.binding.LIB.star_attn_decode(ctypes.byref(sh), p, p, p, p, p, 1, p, 0, V(ws) if ws else None,
                                          ws_bytes, None)


def test_attention_argument_errors(P):
    """Attention calls reject bad shapes, laws, dtypes and pointers on the
    host (fake pointers are never dereferenced)."""
    err = {v: k for k, v in P.binding.STATUS_NAMES.items()}
    assert _raw_attn_fwd(P, _attn_shape(P, law=3)) == err["STAR_ERR_UNSUPPORTED"]  # graph law
    assert _raw_attn_fwd(P, _attn_shape(P, law=7)) == err["STAR_ERR_ARG"]
    assert _raw_attn_fwd(P, _attn_shape(P, head_dim=96, q=2)) == err["STAR_ERR_UNSUPPORTED"]
    assert _raw_attn_fwd(P, _attn_shape(P, q=3)) == err["STAR_ERR_UNSUPPORTED"]    # 64 % 3
    assert _raw_attn_fwd(P, _attn_shape(P, q=16)) == err["STAR_ERR_UNSUPPORTED"]   # m = 4
    assert _raw_attn_fwd(P, _attn_shape(P, q=8, law=2)) == err["STAR_ERR_UNSUPPORTED"]  # tensor power q = 8
    assert _raw_attn_fwd(P, _attn_shape(P, n_kv_heads=3)) == err["STAR_ERR_SHAPE"]
    assert _raw_attn_fwd(P, _attn_shape(P, batch=-1)) == err["STAR_ERR_SHAPE"]
    assert _raw_attn_fwd(P, _attn_shape(P), dt=0) == err["STAR_ERR_DTYPE"]
    assert _raw_attn_fwd(P, _attn_shape(P), ot=5) == err["STAR_ERR_DTYPE"]
    assert _raw_attn_fwd(P, _attn_shape(P), ptrs=None) == err["STAR_ERR_ARG"]
    assert _raw_attn_fwd(P, _attn_shape(P), ptrs=24) == err["STAR_ERR_ALIGN"]
    assert _raw_attn_fwd(P, _attn_shape(P), lse=18) == err["STAR_ERR_ALIGN"]
    assert _raw_attn_fwd(P, _attn_shape(P, batch=0)) == 0                    # no-op
    assert _raw_attn_fwd(P, _attn_shape(P, seq_len=0), ptrs=None) == 0
    need = P.star_attn_decode_workspace_bytes(P.AttnShape(2, 100, 4, 2, 64, 4))
    # two chunks of 128 positions, 4 heads, 2 sequences: 64 features + (max, sum)
    assert need >= 2 * 4 * 1 * (64 + 2) * 4
    assert P.star_attn_decode_workspace_bytes(P.AttnShape(2, 100, 4, 2, 64, 4, "graph")) == 0
    assert _raw_attn_dec(P, _attn_shape(P), ws_bytes=need - 1) == err["STAR_ERR_WORKSPACE"]
    assert _raw_attn_dec(P, _attn_shape(P), ws=None) == err["STAR_ERR_WORKSPACE"]
    assert _raw_attn_dec(P, _attn_shape(P), ptr=8) == err["STAR_ERR_ALIGN"]
    assert _raw_attn_dec(P, _attn_shape(P, seq_len=0)) == err["STAR_ERR_SHAPE"]
    assert _raw_attn_dec(P, _attn_shape(P, batch=0)) == 0


def test_attention_binding_refuses_bad_tensors(P):
    import torch
    sh = P.AttnShape(1, 8, 2, 1, 64, 2)
    Q = torch.zeros((1, 8, 2, 64), dtype=torch.bfloat16)
    K = torch.zeros((1, 8, 1, 64), dtype=torch.bfloat16)
    plan = torch.zeros(64, dtype=torch.uint8)
    with pytest.raises(ValueError):
        P.star_attn_fwd(sh, plan, Q, K[:, :4], K)               # wrong shape
    with pytest.raises(TypeError):
        P.star_attn_fwd(sh, plan, Q.float(), K, K)              # wrong dtype
    with pytest.raises(ValueError):
        P.star_attn_fwd(sh, plan, Q, K, K)                      # CPU tensors
    with pytest.raises(ValueError):
        P.star_attn_decode(sh, torch.zeros(8, dtype=torch.int32), torch.ones(1, dtype=torch.int32),
                           torch.zeros((1, 2, 64), dtype=torch.bfloat16), K, K)
