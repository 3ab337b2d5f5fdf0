"""Host-side pieces of bench.py: the algorithmic work formulas, the latency fit, the
schedule report fed by a latency curve, and the hash-gated readers of committed profiles."""
import math

import numpy as np
import pytest

import bench
from paper_2608_26523_amd import workloads as W


def test_chunk_flops_counts_visible_pairs():
    w = W.get("gqa")
    # one segment of C queries at prefix p: C*p + C*(C+1)/2 pairs, two GEMMs of (dqk + dv)
    for c in range(W.num_chunks(w)):
        _, cu, _, pre = W.chunk_segments(w, c)
        C, p = int(cu[-1]), int(pre[0])
        f, pairs = bench.chunk_flops(w, cu, pre)
        assert pairs == C * p + C * (C + 1) // 2
        assert f == 2.0 * w.hq * (w.dqk + w.dv) * pairs
    # brute force on a small packed chunk
    cu, pre = np.array([0, 3, 3, 8]), np.array([5, 0, 2])
    want = sum(p + r + 1 for (s0, s1, p) in ((0, 3, 5), (3, 3, 0), (3, 8, 2)) for r in range(s1 - s0))
    assert bench.chunk_flops(w, cu, pre)[1] == want


def test_chunk_bytes_formula():
    w = W.get("mla")
    _, cu, _, pre = W.chunk_segments(w, 0)
    C = int(cu[-1])
    want = C * w.hkv * (w.dqk + w.dv) * 2 + C * w.hq * w.dqk * 2 + C * w.hq * w.dv * 2 + C * w.hq * 4
    assert bench.chunk_bytes(w, cu, pre) == want


def test_fit_line_recovers_a_line():
    xs = list(range(8))
    fit = bench.fit_line(xs, [0.19 + 0.237 * x for x in xs])
    assert fit["a_ms"] == pytest.approx(0.19) and fit["b_ms"] == pytest.approx(0.237)
    assert fit["r2"] == pytest.approx(1.0)
    assert fit["b_over_a"] == pytest.approx(0.237 / 0.19)
    assert bench.fit_line([0], [1.0]) is None


def test_schedule_report_on_a_linear_curve():
    # Eq. 2 with t = 1: VPP makespan (N+1)^2, CPP N(N+3) (closed forms pinned in
    # tests/test_schedule_cpu.py), packing strictly shortens two back-to-back requests
    n = 6
    rep = bench.schedule_report([float(k + 1) for k in range(n)])
    assert rep["vpp"]["makespan_ms"] == pytest.approx((n + 1) ** 2)
    assert rep["cpp"]["makespan_ms"] == pytest.approx(n * (n + 3))
    assert rep["vpp_async_packed_2req"]["makespan_ms"] < rep["vpp_async_2req"]["makespan_ms"]
    assert rep["vpp"]["bubble_ratio"] < rep["cpp"]["bubble_ratio"]


def test_profile_readers_are_hash_gated(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_bytes(b"kernel source")
    import hashlib
    sha = hashlib.sha256(b"kernel source").hexdigest()[:16]
    traffic = tmp_path / "t.md"
    traffic.write_text("x\n    traffic gqa %s 12345\n    traffic mla deadbeefdeadbeef 7\n"
                       "    traffic_chunk gqa %s 0 100\n    traffic_chunk gqa %s 1 250\n"
                       "    traffic_chunk mla deadbeefdeadbeef 0 9\n" % (sha, sha, sha))
    mfma = tmp_path / "m.md"
    mfma.write_text("    mfma gqa %s 0.5000 1800\n" % sha)
    monkeypatch.setattr(bench, "KERNEL_SRC", str(src))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(traffic))
    monkeypatch.setattr(bench, "MFMA_FILE", str(mfma))
    assert bench.measured_traffic("gqa") == 12345.0
    assert bench.measured_traffic("mla") is None          # taken on another kernel source
    assert bench.measured_traffic_chunks("gqa") == {0: 100.0, 1: 250.0}
    assert bench.measured_traffic_chunks("mla") is None
    m = bench.measured_mfma("gqa")
    assert m["busy"] == 0.5 and m["clock_mhz"] == 1800.0
    assert m["busy_vs_peak_clock"] == pytest.approx(0.5 * 1800 / 2400)
    # 256 CUs x 4096 flop per clock: 2.5 PFLOP/s at 2.4 GHz
    assert m["peak_at_clock_tflops"] == pytest.approx(2516.6 * 1800 / 2400, abs=0.1)
    assert bench.measured_mfma("mla") is None


def test_committed_profiles_match_the_kernel_source():
    """The committed summaries were taken on the kernel source that is in the tree."""
    assert bench.measured_traffic("gqa") is not None and bench.measured_traffic("mla") is not None
    assert bench.measured_mfma("gqa") is not None and bench.measured_mfma("mla") is not None
    from paper_2608_26523_amd import workloads as W
    for name in ("gqa", "mla"):
        tc = bench.measured_traffic_chunks(name)
        assert tc is not None and sorted(tc) == list(range(W.num_chunks(W.get(name))))
