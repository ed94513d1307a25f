"""Host-side checks of bench.py (no GPU): the one-GPU contract, the source
digest that ties committed profiles to the kernel sources, and the internal
consistency of the committed profile summaries it reports from."""
import importlib.util
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def load_bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_source_digest_ignores_comments_and_layout(tmp_path, monkeypatch):
    bench = load_bench()
    (tmp_path / "a.hip").write_text("int f(int x) {\n  return x + 1;  // one\n}\n/* block\n comment */\n")
    (tmp_path / "b.hip").write_text("int  f(int x) { return x + 1; }\n")
    (tmp_path / "c.hip").write_text("int f(int x) { return x + 2; }\n")
    monkeypatch.setattr(bench, "CSRC", str(tmp_path))
    assert bench.source_digest(("a.hip",)) == bench.source_digest(("b.hip",))
    assert bench.source_digest(("a.hip",)) != bench.source_digest(("c.hip",))


def test_gating_range_matches_the_header():
    # the bench sends gating beyond the f16 chain's stated range to the
    # two-term chain, and beyond that to the float32 path; the ranges are the
    # ones include/mol.h states
    bench = load_bench()
    text = open(os.path.join(ROOT, "include", "mol.h")).read()
    found = re.findall(r"entries\s+\*?\s*of\s+\*?\s*RMS up to ([0-9]+(?:\.[0-9]+)?)", text)
    assert len(found) == 2, "include/mol.h states the f16 and the two-term chains' gating ranges"
    assert float(found[0]) == pytest.approx(bench.F32_GATING_STD)
    assert float(found[1]) == pytest.approx(bench.X2_GATING_STD)


def test_issue_floor_summary_is_consistent():
    # floors follow from the per-wave-step times and the wave-steps per SIMD;
    # the fraction of peak from the floor and the scan's flops
    bench = load_bench()
    path = os.path.join(ROOT, "profiles", "issue_floor_k_mol_fused_exact_1m.txt")
    rows = {}
    kv = {}
    for line in open(path):
        if line.startswith("#"):
            continue
        if ":" in line:
            k, v = line.split(":", 1)
            kv[k.strip()] = float(v)
        elif line.split() and line.split()[0].isdigit():
            f = line.split()
            rows[int(f[0])] = [float(x) for x in f[1:]]
    steps = (1024 // 2) * (1 << 20) // 16 // 1024
    flops = 1024 * (1 << 20) * (2 * 64 * 64 + 4 * 64 * 64)
    for w, (mfma, vec, inter, phased, full, mix_ms, full_ms, full_frac) in rows.items():
        assert full_ms == pytest.approx(full * steps / 1e6, rel=2e-3)
        assert mix_ms == pytest.approx(min(inter, phased) * steps / 1e6, rel=2e-3)
        assert full_frac == pytest.approx(flops / (full_ms / 1e3) / 1e12 / bench.PEAK_BF16_TFLOPS, rel=2e-3)
        assert mfma <= inter and vec <= inter and inter <= full
        assert kv[f"full_stream_floor_ms_w{w}"] == pytest.approx(full_ms, rel=1e-3)
    assert int(kv["kernel_waves_per_simd"]) == 2


def test_fused_profiles_parse_when_current():
    # while the committed summaries carry the current sources' digest the
    # bench reports them; each then holds every field it reads
    bench = load_bench()
    counters = bench.measured_counters("exact_1m")
    traffic = bench.measured_traffic("exact_1m")
    floor = bench.measured_issue_floor("exact_1m")
    if counters is None:
        assert floor is None
        pytest.skip("profiles taken on other kernel sources: the bench reports none of them")
    assert 0.0 < counters["mfma_busy_frac"] < 1.0 and 0.0 < counters["simd_busy_frac"] <= 1.0
    assert traffic is not None and traffic > 1e9
    assert floor is not None and floor["full_stream_floor_ms"] >= floor["mix_floor_ms"]
