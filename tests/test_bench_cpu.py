"""bench.py's accounting on the CPU: the gate/up roofline entry, the
algorithmic bytes of the memory-bound kernel classes and the use of the
committed counter summary.  Expected values are worked out by hand for small
shapes (the arithmetic is in the comments)."""
import hashlib
import json
import os
import sys
from types import SimpleNamespace

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _cfg(**kw):
    base = dict(H=256, F=512, E=8, k=2, dtype="bf16")
    base.update(kw)
    return SimpleNamespace(**base)


def test_gateup_roofline_hbm_bound():
    # 100 pairs, 3 groups, H = 256, F = 512, bf16, 1 ms over 2 launches:
    #   FLOP  = 4 * 256 * 512 * 100                     = 52,428,800
    #   bytes = 3 * (2 * 512 * 256 * 2) + 100 * (256 + 512) * 2
    #         = 1,572,864 + 153,600                      = 1,726,464
    # at the peaks: 52,428,800 / 2.5e15 s = 21 ns < 1,726,464 / 8e12 s = 216 ns
    r = bench.gateup_roofline(_cfg(), pairs=100, groups=3, t_s=1e-3, launches=2, traffic=None)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["achieved"] == pytest.approx(1.726464)
    assert r["frac"] == pytest.approx(1.726464 / 8000.0)
    assert r["hbm_frac"] == pytest.approx(r["frac"])
    assert r["mfma_frac"] == pytest.approx(0.0524288 / 2500.0)
    assert r["algorithmic_flop_per_launch"] == pytest.approx(26_214_400)
    assert r["algorithmic_bytes_per_launch"] == pytest.approx(863_232)
    assert r["avg_launch_ms"] == pytest.approx(0.5)
    assert r["time_at_hbm_peak_ms"] == pytest.approx(1_726_464 / 8e12 * 1e3 / 2)
    assert r["traffic"] is None


def test_gateup_roofline_compute_bound_and_fp32():
    # 10,000 pairs of H = F = 1024 in one group:
    #   FLOP  = 4 * 1024 * 1024 * 10,000                = 41,943,040,000
    #   bytes = 2 * 1024 * 1024 * 2 + 10,000 * 2048 * 2 = 45,154,304
    # 16.8 us at 2.5 PFLOP/s > 5.6 us at 8 TB/s: bound by the matrix cores
    r = bench.gateup_roofline(_cfg(H=1024, F=1024), pairs=10_000, groups=1, t_s=1e-3, launches=1,
                              traffic=123)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s" and r["peak"] == 2500.0
    assert r["achieved"] == pytest.approx(41.94304)
    assert r["frac"] == pytest.approx(41.94304 / 2500.0)
    assert r["hbm_frac"] == pytest.approx(45.154304 / 8000.0)
    assert r["traffic"] == 123
    # fp32: 4-byte elements, priced against the fp32 vector peak
    #   bytes = 2 * 1024 * 1024 * 4 + 10,000 * 2048 * 4 = 90,308,608
    r = bench.gateup_roofline(_cfg(H=1024, F=1024, dtype="f32"), pairs=10_000, groups=1, t_s=1e-3,
                              launches=1, traffic=None)
    assert r["bound"] == "alu" and r["peak"] == pytest.approx(157.3)
    assert r["kernel"] == "grouped_gemm_f32<gate/up>"
    assert r["hbm_frac"] == pytest.approx(90.308608 / 8000.0)


def test_kernel_algorithmic_bytes():
    # H = 256, F = 512, E = 8, k = 2, bf16; 10 tokens, 20 pairs, 3 groups,
    # 2 routing launches:
    #   route   10 * (4*256 + 2*256 + 4*8 + 8*2) + 2 * 8*256*2 = 15,840 + 8,192
    #   gather  (10 + 20) * 256 * 2
    #   combine 20 * (256*2 + 8) + 10 * 8 * 256 = 10,400 + 20,480
    #   down    3 * 512*256*2 + 20 * (512 + 256) * 2 = 786,432 + 30,720
    b = bench.kernel_algorithmic_bytes(_cfg(), tokens=10, pairs=20, groups=3, route_launches=2)
    assert b == {"route_logits": 24_032, "perm_gather": 15_360, "combine": 30_880, "down": 817_152}


def test_measured_traffic_follows_the_kernel_source(tmp_path, monkeypatch):
    src = tmp_path / "paper_2608_07964_amd" / "csrc"
    src.mkdir(parents=True)
    (src / "gemm.hip").write_bytes(b"// kernel source\n")
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    sha = hashlib.sha256(b"// kernel source\n").hexdigest()[:16]
    assert bench.gemm_source_hash() == sha
    path = tmp_path / "profiles" / "gateup_traffic_demo.json"
    assert bench.measured_traffic("demo") is None                       # no summary
    path.write_text(json.dumps({"gemm_source_sha256_16": sha, "hbm_bytes_per_launch": 42}))
    assert bench.measured_traffic("demo") == 42
    path.write_text(json.dumps({"gemm_source_sha256_16": "0" * 16, "hbm_bytes_per_launch": 42}))
    assert bench.measured_traffic("demo") is None                       # taken on another source
