"""CPU checks of the benchmark's host logic (no GPU needed)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


@pytest.mark.parametrize("name,stage", [
    ("void nsg::k_fwd_a<512, 8, false>(float const*, ...)", "fft_fwd_a"),
    ("void nsg::k_pass_b<512, 8, false>(...)", "fft_fwd_b"),
    ("void nsg::k_pass_b<512, 8, true>(...)", "fft_inv_b"),
    ("void nsg::k_inv_a<512, 8>(...)", "fft_inv_a_overlap_add"),
    ("void nsg::k_band_analysis<256, 8>(...)", "band_analysis_256x8"),
    ("void nsg::k_band_synthesis<1024, 16>(...)", "band_synthesis_1024x16"),
    ("void nsg::k_big_a<512, 8>(nsg::BigArgs, ...)", "huge_band_columns"),
    ("void nsg::k_big_b<512, 8>(nsg::BigArgs, ...)", "huge_band_rows"),
    ("nsg::k_ola(float const*, ...)", "sliced_overlap_add"),
    ("__amd_rocclr_copyBuffer", None),
])
def test_profiler_kernel_names_map_to_stages(name, stage):
    assert bench.stage_of_kernel(name) == stage


def test_traffic_is_null_for_other_sources(tmp_path, monkeypatch):
    # counters taken on other kernel sources are not reported
    current = bench.kernel_source_hash()
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "traffic_x.json").write_text(json.dumps(
        {"source_hash": "0" * 16, "kernels": {"k": {"hbm_bytes_per_launch": 1.0}}}))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: current)
    assert bench.traffic_from_profiles("x", "k") is None
    (prof / "traffic_x.json").write_text(json.dumps(
        {"source_hash": current, "kernels": {"k": {"hbm_bytes_per_launch": 5.0}}}))
    assert bench.traffic_from_profiles("x", "k") == 5.0


def test_counted_step_bytes_sums_every_launch(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "traffic_x.json").write_text(json.dumps(
        {"source_hash": "h", "kernels": {"a": {"hbm_bytes_per_launch": 2.0},
                                         "b": {"hbm_bytes_per_launch": 3.0}}}))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "h")
    assert bench.counted_step_bytes("x", ["a", "b", "a"]) == 7.0
    # a launch without counters makes the step figure unknown
    assert bench.counted_step_bytes("x", ["a", "c"]) is None


def test_cpu_baseline_reports_parity_of_the_given_outputs():
    # the oracle leg compares the outputs it is handed with its own; a
    # perturbed copy of the oracle's result shows up at the planted size
    import numpy as np
    import oracle
    import workloads
    w = workloads.WORKLOADS["tiny"]
    x = np.random.default_rng(0).standard_normal((1, w.n_samples)).astype(np.float32)
    lay = oracle.build_layout(*w.plan_args)
    c = oracle.analyse(lay, x)
    xr = oracle.synthesise(lay, c)
    r = bench.cpu_baseline(w, x, target_s=0.01, gpu_c=c * (1 + 1e-3), gpu_x=xr)
    assert r["kind"] == "oracle" and r["parity"]["signals"] == 1
    assert abs(r["parity"]["coeffs_rel_l2_max"] - 1e-3) < 1e-9
    assert r["parity"]["roundtrip_rel_l2_max"] < 1e-12


def test_source_hash_ignores_comments_and_layout():
    a = 'int f(int x) { return x + 1; } // one\nconst char* s = "a // b";'
    b = '/* doc */\nint f(int x) {\n    return x + 1;   // plus one\n}\nconst char* s = "a // b";'
    assert bench.strip_c_comments(a) == bench.strip_c_comments(b)
    # code and string literals still count
    assert bench.strip_c_comments(a) != bench.strip_c_comments(a.replace("+ 1", "+ 2"))
    assert bench.strip_c_comments(a) != bench.strip_c_comments(a.replace('"a // b"', '"a // c"'))


@pytest.mark.parametrize("label", ["stress", "train", "long_full", "long_sliced"])
def test_stage_elements_count_coefficients_and_points(label):
    # the counter summary's per-element figures: the band kernels of one
    # direction produce every coefficient of the step once, the FFT passes
    # transform L points per signal
    import workloads
    from paper_2609_29119_amd import nsgcqt as nb
    e = bench.stage_elements(label)
    w = workloads.WORKLOADS[label.split("_")[0]]
    if label == "long_sliced":
        p, b = nb.Plan.sliced(w.fs, w.fmin, w.fmax, w.bins_per_octave, w.slice_len, 16, device=False), 16
    else:
        b = 1 if w.slice_len else w.batch
        p = nb.Plan(*w.plan_args, batch=b, device=False)
    an = sum(v for k, v in e.items() if k.startswith("band_analysis"))
    if label != "long_full":     # the full-length long plan also has huge bands
        assert an == pytest.approx(p.n_coeffs * b, rel=1e-9)
    assert e["fft_fwd_a"] == pytest.approx(p.info.packed_len * b, rel=1e-12)
    assert e["fft_inv_a_overlap_add" if label != "train" else "fft_fwd_b"] == pytest.approx(
        p.info.packed_len * b, rel=1e-9)
