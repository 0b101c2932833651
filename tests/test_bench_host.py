"""Host-side logic of bench.py (no GPU): the roofline peaks, the rotated
buffer sets and their assignment to streams, the committed-traffic lookup
and its source hash, and the one-GPU guard."""
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
    for case in cases:
        assert bench.sets_for(case, 5) % bench.N_STREAMS == 0, case.name


@pytest.mark.parametrize("n_sets,n_streams", [(8, 2), (6, 2), (6, 3),
                                              (12, 4), (7, 1)])
@pytest.mark.parametrize("first,steps", [(0, 20), (5, 20), (3, 7), (20, 1)])
def test_steps_that_share_buffers_share_a_stream(n_sets, n_streams, first,
                                                 steps):
    bench.check_sets_streams(n_sets, n_streams)
    streams = [bench.stream_of(j, steps, n_streams) for j in range(steps)]
    assert streams[0] == 0                        # start event's stream
    for j in range(steps):
        for k in range(j + 1, steps):
            if (first + j) % n_sets == (first + k) % n_sets:
                assert streams[j] == streams[k]
            if k == j + 1 and n_streams > 1:
                assert streams[j] != streams[k]   # neighbours alternate


def test_sets_not_a_multiple_of_the_streams_are_refused():
    with pytest.raises(ValueError):
        bench.check_sets_streams(7, 2)
    bench.check_sets_streams(0, 2)                # fresh outputs only


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
