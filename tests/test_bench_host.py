"""Host-side logic of bench.py (no GPU): the roofline peaks, the rotated
buffer sets, the committed-traffic lookup and its source hash, and the
one-GPU guard."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_1810_11066_amd import workloads as wl  # noqa: E402


@pytest.mark.parametrize("a,w,tops", [(1, 1, 1258.3), (2, 1, 629.1),
                                      (2, 2, 314.6), (3, 3, 139.8)])
def test_popcount_roofline(a, w, tops):
    # 256 CUs x 64 lanes x 2.4 GHz lane-ops, an AND and a popcount per
    # 32 binary MACs, A*W binary MACs per A-bit x W-bit MAC
    assert bench.popcount_roofline_tops(a, w) == pytest.approx(tops, abs=0.05)


def test_strip_comments_keeps_code_and_literals():
    src = ('int a = 1; // one\n'
           '/* block\n comment */ const char* s = "x // not a comment";\n'
           "char c = '/'; const char* t = \"q\\\"//\"; int b;\n")
    got = bench.strip_comments(src)
    assert got == ('int a = 1; const char* s = "x // not a comment"; '
                   "char c = '/'; const char* t = \"q\\\"//\"; int b;")
    # comments and layout do not change the result, code does
    assert bench.strip_comments("int  a=1;\n// note\n") == \
        bench.strip_comments("int a=1; /* other note */")
    assert bench.strip_comments("int a=1;") != bench.strip_comments("int a=2;")


def test_committed_traffic_follows_the_code(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    name = "conv2d_some_workload_traffic.md"
    (tmp_path / name).write_text(
        "kernel_source_sha256: %s\nhbm_bytes_per_launch: 12345\n"
        % bench.kernel_source_hash())
    assert bench.committed_traffic("some_workload") == 12345.0
    (tmp_path / name).write_text(
        "kernel_source_sha256: 0000000000000000\nhbm_bytes_per_launch: 1\n")
    assert bench.committed_traffic("some_workload") is None
    assert bench.committed_traffic("missing_workload") is None


def test_rotated_sets_pass_twice_the_infinity_cache():
    cases = ([wl.config2(), wl.config3()] + wl.config4() +
             wl.config4(batch=16) + wl.config5() + wl.encodings() +
             wl.bitwidth_sweep())
    for case in cases:
        n = bench.sets_for(case, 6)
        assert 6 <= n <= 256
        pre, _ = bench.case_bytes(case)
        if isinstance(case, wl.DenseCase):
            out = case.m * case.n * 4
        else:
            out = case.n * case.oh * case.ow * case.oc * 4
        if n < 256:
            assert n * (pre + out) >= 512 * 10**6, case.name
    assert bench.sets_for(wl.config2(), 6) == 8


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
