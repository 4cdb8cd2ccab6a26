"""Host-side logic of bench.py (no GPU): the algorithmic byte counts behind the
roofline, and the calibration of the rocprofv3 traffic counters."""

import csv
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads  # noqa: E402


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_step_bytes_follow_the_per_edge_formula(name):
    """The three kernels together move 4 E (5 U d1 + 3 U + 3 d2) + 16 N U d2 bytes
    (x read twice, out, g and grad_x once each; w twice and grad_w; Y twice and
    grad_Y; env written and read twice, grad_env written), plus row_ptr and the
    path weights."""
    g = workloads.make_graph(name)
    cfg = g.config
    d1, d2, n_paths = workloads.dims(cfg.lmax, cfg.full_parity)
    U, N, E = cfg.U, g.n_atoms, g.n_edges
    b = bench.algorithmic_bytes(cfg, N, E)
    small = (N + 1) * 8 + n_paths * U * 4
    total = b["env_embed"] + b["tp_forward"] + b["tp_backward"]
    # env_embed reads row_ptr only; the forward and the backward also read the path weights
    assert total == 4 * E * (5 * U * d1 + 3 * U + 3 * d2) + 16 * N * U * d2 + (N + 1) * 8 + 2 * small


def test_headline_bytes_per_edge():
    """About 24.1 KB per edge at U = 64, lmax 2 with full parity and mean degree 52.4
    (4 (5 U d1 + 3 U + 3 d2) + 16 U d2 / degree)."""
    d1, d2, _ = workloads.dims(2, True)
    per_edge = 4 * (5 * 64 * d1 + 3 * 64 + 3 * d2) + 16 * 64 * d2 / 52.4
    assert (d1, d2) == (18, 9)
    assert abs(per_edge - 24092) < 1


def test_layer_bytes():
    cfg = workloads.CONFIGS["medium_layer"]
    d1, d2, _ = workloads.dims(cfg.lmax, cfg.full_parity)
    L, UD = cfg.extra["L"], cfg.U * d1
    b = bench.layer_algorithmic_bytes(cfg, 1000)
    # forward: h, V, Y in; h', V' out.  backward: h, V, Y, dh', dV' in; dh, dV, dY out
    assert b["forward"] == 4 * 1000 * (L + UD + d2 + L + UD)
    assert b["backward"] == 4 * 1000 * (L + UD + d2 + L + UD + L + UD + d2)


def test_source_digest_is_stable():
    a, b = bench.kernel_source_digest(), bench.kernel_source_digest()
    assert a == b and len(a) == 16 and int(a, 16) >= 0


def _write_counters(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Value"])
        w.writeheader()
        for name, value in rows:
            w.writerow({"Kernel_Name": name, "Counter_Value": value})


def test_pmc_summary_calibrates_and_selects_the_inference_backward(tmp_path, monkeypatch):
    """Each counter is scaled by what it reads for the 4 GiB copy; only the inference
    backward's dispatches (template flag false) are averaged, not the training ones."""
    copy_kib = (4 << 30) / 1024
    inf = "void (anonymous namespace)::tp_backward_kernel<TPCore<1, false>, 16, false, 16>(long const*)"
    train = "void (anonymous namespace)::tp_backward_kernel<TPCore<1, false>, 16, true, 4>(long const*)"
    fetch = tmp_path / "fetch.csv"
    write = tmp_path / "write.csv"
    # fetch counts half of the copy's bytes, write all of them
    _write_counters(fetch, [("__amd_rocclr_copyBuffer", copy_kib / 2), (inf, 100.0), (inf, 300.0), (train, 1e9)])
    _write_counters(write, [("__amd_rocclr_copyBuffer", copy_kib), (inf, 50.0), (inf, 50.0), (train, 1e9)])
    out = tmp_path / "traffic.json"
    bench.pmc_summary(str(fetch), str(write), "tiny", str(out))
    rec = json.loads(out.read_text())
    assert rec["dispatches"] == 2
    assert rec["fetch_kib_per_dispatch"] == 200.0 and rec["write_kib_per_dispatch"] == 50.0
    assert rec["copy_calibration"]["fetch_scale"] == 2.0 and rec["copy_calibration"]["write_scale"] == 1.0
    assert rec["traffic_bytes_per_launch"] == (200.0 * 2 + 50.0) * 1024
    g = workloads.make_graph("tiny")
    assert rec["algorithmic_bytes_per_launch"] == bench.algorithmic_bytes(g.config, g.n_atoms, g.n_edges)["tp_backward"]
    # the record is used only while the kernel sources and the workload match
    monkeypatch.setattr(bench, "PROFILE_TRAFFIC", str(out))
    assert bench.measured_traffic("tiny") == rec["traffic_bytes_per_launch"]
    assert bench.measured_traffic("headline") is None
    rec["kernel_source_digest"] = "0" * 16
    out.write_text(json.dumps(rec))
    assert bench.measured_traffic("tiny") is None
