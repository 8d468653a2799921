"""Host-side checks of bench.py's contract (no GPU needed)."""

import importlib.util
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench_module():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_key_ignores_comments_only(tmp_path):
    b = _bench_module()
    src = tmp_path / "k.hip"
    src.write_text("int f(int x) {  // doubles\n  return 2 * x;\n}\n")
    b.GEMM_SRCS = [str(src)]
    h0 = b.gemm_src_hash()
    src.write_text("// a new comment\nint f(int x) {  // twice x\n\n  return 2 * x;\n}\n")
    assert b.gemm_src_hash() == h0
    src.write_text("int f(int x) {\n  return 3 * x;\n}\n")
    assert b.gemm_src_hash() != h0

