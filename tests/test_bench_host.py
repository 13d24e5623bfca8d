"""Host-side logic of bench.py (no GPU): the kernel names it reports exist in the sources, and
committed traffic counters are used only while the sources they were taken on are unchanged."""
import hashlib
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402


def test_kernel_source_file_maps_kernels_to_their_files():
    assert bench.kernel_source_file("k_accumulate_il<2>") == "k_stream.hip"
    assert bench.kernel_source_file("k_pull<8, 6, true>") == "k_pull.hip"
    assert bench.kernel_source_file("k_digit2") == "k_select.hip"
    assert bench.kernel_source_file("k_no_such_kernel") is None


@pytest.mark.parametrize("layout", ["interleaved", "worker_major"])
@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_stage_kernels_name_existing_kernels(name, layout):
    # a renamed or removed kernel left in the stage lists would silently void the roofline's
    # traffic figure; every name must resolve to a __global__ definition
    w = synth.WORKLOADS[name]
    for stage, names in bench.stage_kernels(w, layout).items():
        for n in names:
            assert bench.kernel_source_file(n) is not None, f"{stage}: {n} is not defined in csrc"


def _profile(tmp_path, w, layout, hashes, traffic):
    d = tmp_path / "profiles"
    d.mkdir(exist_ok=True)
    lines = [f"    source_sha256[{f}]: {h}" for f, h in hashes.items()]
    lines += [f"    traffic: {n} | {v:.0f}" for n, v in traffic.items()]
    (d / f"traffic_gs_step_{w.name}_{layout}.md").write_text("\n".join(lines) + "\n")


def _current_hashes():
    out = {}
    for f in sorted(os.listdir(bench.CSRC)):
        with open(os.path.join(bench.CSRC, f), "rb") as fh:
            out[f] = hashlib.sha256(fh.read()).hexdigest()
    return out


def test_traffic_used_while_sources_match(tmp_path, monkeypatch):
    w = synth.WORKLOADS["laplace53-d25.6M-P8"]
    acc = bench.stage_kernels(w)["accumulate"][0]
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    _profile(tmp_path, w, "interleaved", _current_hashes(), {acc: 4.096e9})
    assert bench.measured_traffic(w, "accumulate") == pytest.approx(4.096e9)


def test_traffic_dropped_when_a_dependency_changed(tmp_path, monkeypatch):
    w = synth.WORKLOADS["laplace53-d25.6M-P8"]
    acc = bench.stage_kernels(w)["accumulate"][0]
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    # the kernel's own file
    h = _current_hashes()
    h[bench.kernel_source_file(acc)] = "0" * 64
    _profile(tmp_path, w, "interleaved", h, {acc: 4.096e9})
    assert bench.measured_traffic(w, "accumulate") is None
    # a shared launcher/header file
    h = _current_hashes()
    h["gs_api.hip"] = "0" * 64
    _profile(tmp_path, w, "interleaved", h, {acc: 4.096e9})
    assert bench.measured_traffic(w, "accumulate") is None
    # another kernel's file does not matter
    h = _current_hashes()
    h["k_select.hip"] = "0" * 64
    _profile(tmp_path, w, "interleaved", h, {acc: 4.096e9})
    assert bench.measured_traffic(w, "accumulate") == pytest.approx(4.096e9)


def test_traffic_absent_without_profile_or_kernel_entry(tmp_path, monkeypatch):
    w = synth.WORKLOADS["laplace53-d25.6M-P8"]
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic(w, "accumulate") is None
    _profile(tmp_path, w, "interleaved", _current_hashes(), {"k_other": 1.0})
    assert bench.measured_traffic(w, "accumulate") is None


def test_gpu_count_above_one_exits_with_a_message(monkeypatch, capsys):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--gpus", "2"])
    with pytest.raises(SystemExit) as e:
        bench.main()
    assert e.value.code not in (0, None)


def test_cpu_baseline_runs_whole_steps_within_its_bounds():
    # consecutive oracle steps until the minimum time has passed; the rate counts every step
    w = synth.WORKLOADS["t3planted-d65536-P4"]
    r = bench.cpu_baseline(w, synth.gradients(w, 0), budget_s=5.0, min_s=0.2)
    assert r["kind"] == "oracle" and r["cores"] == 1 and r["steps"] >= 1
    assert 0.2 <= r["seconds"] <= 5.0
    assert r["value"] == pytest.approx(r["steps"] * w.P * w.d / r["seconds"], rel=1e-2)


def test_roofline_names_the_co_dominant_stage_furthest_below_peak():
    # two stages within 10% of each other: the one with the lower algorithmic fraction is the
    # dominant kernel, both are listed, and the step fraction is B / t / 8 TB/s
    st = [
        {"stage": "accumulate", "kernel": "a", "mean_ms": 0.66, "bytes_per_launch": 4.096e9, "achieved": 6206.0,
         "frac": 0.776, "traffic": None, "traffic_frac": None},
        {"stage": "sketch", "kernel": "p", "mean_ms": 0.645, "bytes_per_launch": 0.824e9, "achieved": 1277.0,
         "frac": 0.160, "traffic": None, "traffic_frac": None},
        {"stage": "select", "kernel": "s", "mean_ms": 0.14, "bytes_per_launch": 5.2e6, "achieved": 37.0,
         "frac": 0.005, "traffic": None, "traffic_frac": None},
    ]
    r = bench.roofline_of(st, 4_000_000_000, 1.25)
    assert r["stage"] == "sketch" and r["frac"] == 0.160
    assert [e["stage"] for e in r["co_dominant"]] == ["accumulate", "sketch"]
    assert abs(r["step"]["frac"] - 4e9 / 1.25e-3 / 1e9 / 8000.0) < 1e-12
    assert bench.roofline_of([], 1, 1.0) is None


def test_step_bytes_leave_out_the_tables_the_fused_step_never_writes():
    w = synth.WORKLOADS["laplace53-d25.6M-P8"]
    assert bench.step_bytes(w) == 20 * w.P * w.d + 8 * w.r * w.c + 12 * w.P * w.k + 8 * w.k
    assert bench.stage_bytes(w)["merge"] == 0
