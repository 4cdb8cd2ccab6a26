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
    """Each counter is scaled by what it reads for the 4 GiB one-read-one-write
    probe; only the inference backward's dispatches (template flag false) are
    averaged, not the training ones."""
    copy_kib = (4 << 30) / 1024
    inf = "void (anonymous namespace)::tp_backward_kernel<TPCore<1, false>, 16, false, 16>(long const*)"
    train = "void (anonymous namespace)::tp_backward_kernel<TPCore<1, false>, 16, true, 4>(long const*)"
    probe = "void (anonymous namespace)::stream_kernel<1, 4>(float const*)"
    probe_read = "void (anonymous namespace)::stream_kernel<0, 4>(float const*)"
    fetch = tmp_path / "fetch.csv"
    write = tmp_path / "write.csv"
    # fetch counts half of the probe's bytes, write all of them
    _write_counters(fetch, [(probe, copy_kib / 2), (probe, copy_kib / 2), (probe_read, 1.0), (inf, 100.0),
                            (inf, 300.0), (train, 1e9)])
    _write_counters(write, [(probe, copy_kib), (probe, copy_kib), (probe_read, 5.0), (inf, 50.0), (inf, 50.0),
                            (train, 1e9)])
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    bench.pmc_summary(str(fetch), str(write), "tiny", "tp_backward")
    out = tmp_path / "tp_backward_tiny_traffic.json"
    rec = json.loads(out.read_text())
    assert rec["dispatches"] == 2
    assert rec["fetch_kib_per_dispatch"] == 200.0 and rec["write_kib_per_dispatch"] == 50.0
    assert rec["calibration"]["fetch_scale"] == 2.0 and rec["calibration"]["write_scale"] == 1.0
    assert rec["traffic_bytes_per_launch"] == (200.0 * 2 + 50.0) * 1024
    g = workloads.make_graph("tiny")
    assert rec["algorithmic_bytes_per_launch"] == bench.algorithmic_bytes(g.config, g.n_atoms, g.n_edges)["tp_backward"]
    # the record is used only while the kernel sources and the workload match
    assert bench.measured_traffic("tp_backward", "tiny") == rec["traffic_bytes_per_launch"]
    assert bench.measured_traffic("tp_backward", "headline") is None
    rec["kernel_source_digest"] = "0" * 16
    out.write_text(json.dumps(rec))
    assert bench.measured_traffic("tp_backward", "tiny") is None


def test_pmc_patterns_select_their_kernels():
    import re
    names = {
        "tp_backward": ["void (anonymous namespace)::tp_backward_kernel<TPCore<2, true>, 64, false, 16>(long const*)",
                        "void (anonymous namespace)::tp_backward_kernel<TPCore<3, true>, 128, false, 8>(long const*)"],
        "tp_forward": ["void (anonymous namespace)::tp_forward_kernel<TPCore<2, true>, 64, 16>(long const*)",
                       "void (anonymous namespace)::tp_matrix_kernel<TPCore<3, true>, 128, TPMFwd<3, true> >(long)"],
        "tp_mfma_bwd": ["void (anonymous namespace)::tp_mfma_bwd_kernel<true, 128, true>(long, long const*)"],
    }
    for key, pattern in bench.TRAFFIC_KERNELS.items():
        for other, kernels in names.items():
            for name in kernels:
                assert bool(re.search(pattern, name)) == (key == other), (key, other, name)
    # the training backward at lmax <= 2 and the backward's grad_x matrix kernel are not selected
    for pattern in bench.TRAFFIC_KERNELS.values():
        assert not re.search(pattern, "void (anonymous namespace)::tp_backward_kernel<TPCore<2, true>, 64, true, 4>(long)")
        assert not re.search(pattern, "void (anonymous namespace)::tp_matrix_kernel<TPCore<3, true>, 64, "
                                      "TPMBwdX<3, true> >(long)")


def test_mfma_bwd_bytes():
    g = workloads.make_graph("tiny")
    cfg = workloads.CONFIGS["high_order"]
    d1, d2, P = workloads.dims(cfg.lmax, cfg.full_parity)
    N, E = 10, 1000
    # x, g read and grad_x written; env read and grad_env written; row_ptr and the path weights
    # (the kernel's per-wave path-weight rows, well under a megabyte, are left out)
    assert bench.mfma_bwd_bytes(cfg, N, E) == (4 * (3 * E * cfg.U * d1 + 2 * N * cfg.U * d2)
                                               + (N + 1) * 8 + 4 * P * cfg.U)
    del g


def test_cpu_baseline_ranges_cover_the_sample():
    """The oracle's per-process ranges run every center of the sample exactly once."""
    g = workloads.make_graph("tiny")
    x, w, pw, gr = workloads.host_features(g.config, g.n_edges)
    from oracle import tp as otp
    bench._CPU_JOB.update(row_ptr=g.row_ptr, x=x, w=w, Y=g.Y, pw=pw, g=gr,
                          tp=otp.TensorProduct(g.config.lmax, g.config.full_parity))
    try:
        n = g.n_atoms
        assert bench._cpu_range((0, n)) == g.n_edges
        assert bench._cpu_range((0, 10)) + bench._cpu_range((10, n)) == g.n_edges
    finally:
        bench._CPU_JOB.clear()
