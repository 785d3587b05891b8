"""bench.py's host logic (CPU): the one-GPU refusal, launch-string parsing and
the lookup of the headline kernel's HBM traffic from its counter summary."""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}),
                                      ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused(argv, env):
    e = dict(os.environ, **env)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv],
                       capture_output=True, text=True, env=e, timeout=120)
    assert r.returncode == 2, r.stderr
    assert "one GPU" in r.stderr and r.stdout == ""


def test_launch_strings(bench):
    from paper_2502_19405_amd import repops
    assert bench.parse_launch("auto", repops) is None
    assert bench.parse_launch("", repops) is None
    assert bench.parse_launch("simple", repops).kind == repops.LAUNCH_GEMM_SIMPLE
    t = bench.parse_launch("tiled:2", repops)
    assert (t.kind, t.p[0]) == (repops.LAUNCH_GEMM_TILED, 2)
    m = bench.parse_launch("mfma", repops)
    assert (m.kind, m.p[0]) == (repops.LAUNCH_GEMM_MFMA, 0)


def test_traffic_comes_only_from_a_matching_counter_summary(bench, tmp_path, monkeypatch):
    summary = tmp_path / "counters.md"
    summary.write_text("prose\n\ntraffic_bytes_per_launch_dX = 1234567\n"
                       "traffic_bytes_per_launch_dW = 7654321\n"
                       f"kernel_source_sha256 = {bench.kernel_source_sha256()}\n")
    monkeypatch.setattr(bench, "COUNTERS_MD", str(summary))
    assert bench.measured_traffic("auto", "dX") == 1234567.0
    assert bench.measured_traffic("mfma:0", "dW") == 7654321.0
    assert bench.measured_traffic("mfma:1", "dX") is None  # another kernel: no figure
    # A source that differs from the one the counters were taken on voids it.
    src = tmp_path / "gemm_mfma.hip"
    src.write_bytes(open(bench.KERNEL_SOURCES[0], "rb").read() + b"\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCES", [str(src), *bench.KERNEL_SOURCES[1:]])
    assert bench.measured_traffic("auto", "dX") is None


def test_committed_counter_summary_parses(bench):
    """The committed summary, when present, holds both products' figures (at
    least their algorithmic bytes) -- or is stale, in which case bench.py
    reports no traffic rather than a figure for other kernel sources."""
    if not os.path.exists(bench.COUNTERS_MD):
        pytest.skip("no counter summary committed")
    for product, algorithmic in (("dX", 4 * (8192 * 14336 + 4096 * 14336 + 8192 * 4096)),
                                 ("dW", 4 * (8192 * 4096 + 8192 * 14336 + 4096 * 14336))):
        v = bench.measured_traffic("auto", product)
        assert v is None or v >= algorithmic, (product, v)


def test_clock_sampler_reads_the_starred_level(bench, tmp_path):
    f = tmp_path / "pp_dpm_sclk"
    f.write_text("0: 500Mhz\n1: 2187Mhz *\n2: 2400Mhz\n")
    c = bench.ClockSampler()
    c.path = str(f)
    assert c._read() == 2187
    c.samples = [2400, 2100, 2150, 2160, 2170]
    assert c.median() == 2160  # the first quarter (ramp) is left out
    f.write_text("0: 500Mhz\n")
    assert c._read() is None
    c.path = str(tmp_path / "missing")
    assert c._read() is None
