"""Host-side tests of bench.py's readers of the committed counter profiles (no GPU).

The bench line reports HBM traffic, clock and MFMA occupancy from profile summaries only
while the kernel source they were taken on is the current one.  These tests write
summaries of their own and check that values are read when workload and source hash
match, and that a stale, foreign or missing summary yields null.
"""
import bench

WL = "longctx_bf16_T32768_d2880_V201088_P8_ring"


def _summary(path, sha, workload=WL, extra=()):
    lines = ["# a summary", "", "Values read by bench.py:", "",
             f"- workload: `{workload}`", f"- kernel_source_sha256: `{sha}`"]
    lines += [f"- {k}: `{v}`" for k, v in extra]
    path.write_text("\n".join(lines) + "\n")


def test_traffic_read_while_the_source_hash_matches(tmp_path, monkeypatch):
    p = tmp_path / "traffic.md"
    _summary(p, bench.kernel_source_sha256(),
             extra=[("fwd_kernel_hbm_bytes_per_launch", "6.5e+10"),
                    ("bwd_stage_kernel_hbm_bytes_per_launch", "5.2e+09")])
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(p))
    assert bench.measured_traffic("fwd_kernel", WL) == 6.5e10
    assert bench.measured_traffic("bwd_stage_kernel", WL) == 5.2e9
    assert bench.measured_traffic("transpose_kernel", WL) is None  # not in the summary
    assert bench.measured_traffic("fwd_kernel", "bf16_T4096_d2880_V201088_P8") is None


def test_stale_or_missing_profile_gives_null(tmp_path, monkeypatch):
    p = tmp_path / "traffic.md"
    _summary(p, "0" * 64, extra=[("fwd_kernel_hbm_bytes_per_launch", "6.5e+10")])
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(p))
    assert bench.measured_traffic("fwd_kernel", WL) is None
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(tmp_path / "absent.md"))
    assert bench.measured_traffic("fwd_kernel", WL) is None


def test_clock_and_occupancy(tmp_path, monkeypatch):
    p = tmp_path / "mfma.md"
    _summary(p, bench.kernel_source_sha256(),
             extra=[("fwd_kernel_clock_ghz", "1.5"), ("fwd_kernel_mfma_busy", "0.75")])
    monkeypatch.setattr(bench, "MFMA_PROFILE", str(p))
    c = bench.measured_clock("fwd_kernel", WL)
    assert c["clock_ghz"] == 1.5 and c["mfma_busy"] == 0.75
    # the nameplate peak is quoted at 2.4 GHz
    assert abs(c["peak_at_clock"] - bench.PEAK_BF16_TFLOPS * 1.5 / 2.4) < 1e-9
    assert bench.measured_clock("bwd_stage_kernel", WL) is None
    _summary(p, "f" * 64, extra=[("fwd_kernel_clock_ghz", "1.5"), ("fwd_kernel_mfma_busy", "0.75")])
    assert bench.measured_clock("fwd_kernel", WL) is None


def test_frac_at_clock(tmp_path, monkeypatch):
    p = tmp_path / "mfma.md"
    _summary(p, bench.kernel_source_sha256(),
             extra=[("fwd_kernel_clock_ghz", "1.5"), ("fwd_kernel_mfma_busy", "0.75")])
    monkeypatch.setattr(bench, "MFMA_PROFILE", str(p))
    roof = {"achieved": 1000.0, "counters": bench.measured_clock("fwd_kernel", WL)}
    bench.add_frac_at_clock(roof, "bf16")
    assert abs(roof["counters"]["frac_at_clock"] - 1000.0 / (bench.PEAK_BF16_TFLOPS * 1.5 / 2.4)) < 1e-12
    roof = {"achieved": 1000.0, "counters": None}
    bench.add_frac_at_clock(roof, "bf16")  # no profile for this kernel source: nothing added
    assert roof["counters"] is None


def test_committed_profiles_name_the_default_workload():
    # the committed summaries cover the workload bench.py runs by default
    for path in (bench.TRAFFIC_PROFILE, bench.MFMA_PROFILE):
        text = open(path).read()
        assert f"- workload: `{bench.DEFAULT_WORKLOAD}`" in text
        assert "- kernel_source_sha256: `" in text


def test_more_than_one_gpu_is_refused():
    # one GPU's share of the ring: the benchmark refuses other GPU counts before any GPU work
    import json
    import subprocess
    import sys

    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "exactly one GPU" in line["error"] and line["n_gpus"] == 2
