"""Benchmark: Allegro tensor product forward + backward edges/s on one MI355X.

One step is one pass of the whole hot path over the resident workload:
allegro_env_embed + allegro_tp_forward + allegro_tp_backward (the backward
includes the embedding's VJP), all on one HIP stream, inputs already in HBM.

Workload (default): 20,000 atoms uniform in a periodic cube at 0.1 atoms/A^3
(the number density of liquid water), cutoff 5 A (about 1.05e6 directed edges,
CSR by center), U = 64 channels, lmax = 2 with full parity (d1 = 18, d2 = 9,
30 paths, 274 coupling non-zeros); fp32 features drawn N(0, 1), path weights
N(0, 1/sqrt(30)).  Synthetic data: no dataset of the paper is used.

Prints ONE JSON line.  The roofline object describes the dominant kernel
(tp_backward): algorithmic bytes per launch over its mean duration, measured
with HIP events on the stream the library launches on, against the 8 TB/s
HBM peak and against the rate of a plain streaming kernel of the same access
pattern timed in the same run (stream_probes).  Extra keys:
  high_order      the same step at Table I's large-model shape (lmax 3, 128
                  channels), with its own roofline object;
  large           the headline step on 100,000 atoms at cutoff 6 A (about 9e6
                  edges), with its own roofline object;
  allegro_layer   one whole Allegro layer (forward, and backward with every
                  weight gradient) at the medium model shape of Table I;
  cpu_baseline    the fp64 oracle on bounded samples of the small, headline and
                  high-order workloads, timed before the GPU is touched.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--no-cpu-baseline] [--no-layer] [--no-high-order] [--no-large]
       python bench.py --layer-only
       python bench.py --pmc-summary FETCH_CSV WRITE_CSV --pmc-kernel NAME
                       (after two rocprofv3 --pmc runs; see pmc_summary)
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads  # noqa: E402

METRIC = "Allegro TP fwd+bwd edges/sec at lmax=2, 64 ch; % of HBM (or MFMA) roofline"
HBM_PEAK_GBPS = 8000.0
HOST_SHARE = 16  # host cores that go with one GPU on the MI355X hosts
PROFILES = os.path.join(ROOT, "profiles")
# kernels with committed rocprofv3 traffic records (profiles/<kernel>_<workload>_traffic.json):
# the kernel-name pattern of each
TRAFFIC_KERNELS = {
    "tp_backward": r"tp_backward_kernel<TPCore<\d+,\s*(true|false)>,\s*\d+,\s*false(,\s*\d+)?>",
    "tp_forward": r"tp_(forward|matrix)_kernel<TPCore<\d+,\s*(true|false)>,\s*\d+(,\s*\d+)?(,\s*TPMFwd<[^>]*>\s*)?>",
    "tp_mfma_bwd": r"tp_mfma_bwd_kernel<(true|false),\s*\d+,\s*true>",
}


def traffic_record_path(kernel: str, workload: str) -> str:
    return os.path.join(PROFILES, f"{kernel}_{workload}_traffic.json")
# the sources the kernels are built from, with their build flags
DIGEST_SOURCES = ("paper_2504_16068_amd/csrc/allegro_tp.hip", "paper_2504_16068_amd/csrc/allegro_layer.hip",
                  "paper_2504_16068_amd/csrc/device_common.hpp", "paper_2504_16068_amd/csrc/plan.hpp",
                  "paper_2504_16068_amd/csrc/gen_kernels.cpp", "paper_2504_16068_amd/csrc/cg_builder.cpp",
                  "paper_2504_16068_amd/csrc/cg_builder.hpp", "paper_2504_16068_amd/build.py",
                  "include/allegro_tp.h", "include/allegro_layer.h")


def algorithmic_bytes(cfg, n_atoms: int, n_edges: int):
    """Bytes each call must move at least once (fp32 data, int64 row_ptr).

    env_embed:   read w [E,U] and Y [E,d2]; write env [N,U,d2]
    tp_forward:  read x [E,U,d1] and env; write out [E,U,d1]
    tp_backward: read x, g [E,U,d1], env, w, Y; write grad_x [E,U,d1],
                 grad_env [N,U,d2], grad_w [E,U], grad_Y [E,d2]
    (row_ptr and the path weights add (N+1)*8 and P*U*4 bytes to each.)
    """
    d1, d2, n_paths = workloads.dims(cfg.lmax, cfg.full_parity)
    u = cfg.U
    small = (n_atoms + 1) * 8 + n_paths * u * 4
    env_b = 4 * (n_edges * (u + d2) + n_atoms * u * d2) + (n_atoms + 1) * 8
    fwd_b = 4 * (2 * n_edges * u * d1 + n_atoms * u * d2) + small
    bwd_b = 4 * (n_edges * (3 * u * d1 + 2 * u + 2 * d2) + 2 * n_atoms * u * d2) + small
    return {"env_embed": env_b, "tp_forward": fwd_b, "tp_backward": bwd_b}


def mfma_bwd_bytes(cfg, n_atoms: int, n_edges: int):
    """Algorithmic bytes of the lmax-3 training backward's first kernel (tp_mfma_bwd_kernel):
    read x, g [E,U,d1] and env; write grad_x [E,U,d1] and grad_env [N,U,d2].  Its
    path-weight partial sums (one [U][P] row per round of its waves, 16 rounds
    on a 256-CU device: about 0.6 MB at U = 128) are left out."""
    d1, d2, n_paths = workloads.dims(cfg.lmax, cfg.full_parity)
    u = cfg.U
    return 4 * (3 * n_edges * u * d1 + 2 * n_atoms * u * d2) + (n_atoms + 1) * 8 + n_paths * u * 4


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    for rel in DIGEST_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(key: str, workload: str):
    """HBM bytes per launch from a committed rocprofv3 record, if it was taken on the
    current kernel sources and this workload; else None."""
    path = traffic_record_path(key, workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_digest") != kernel_source_digest() or rec.get("workload") != workload:
        return None
    return rec.get("traffic_bytes_per_launch")


def pmc_summary(fetch_csv: str, write_csv: str, workload: str, key: str):
    """Calibrated HBM traffic of one kernel from two rocprofv3 --pmc runs of this script.

    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are each scaled by what the same
    counter reads for the streaming probe's one-read-one-write kernel over 4 GiB
    (stream_kernel<1, ...>: exactly 4 GiB read and 4 GiB written), so that the
    request-size conventions of the counters cancel out.  Writes the record that
    bench.py reads as roofline.traffic.
    """
    import csv

    def read(path):
        with open(path) as f:
            return list(csv.DictReader(f))

    copy_kib = (4 << 30) / 1024
    pattern = TRAFFIC_KERNELS[key]
    pat = re.compile(pattern)

    def per_launch(rows):
        vals = [float(r["Counter_Value"]) for r in rows if pat.search(r["Kernel_Name"])]
        return sum(vals) / len(vals), len(vals)

    def calibration(rows):
        vals = [float(r["Counter_Value"]) for r in rows if "stream_kernel<1" in r["Kernel_Name"]]
        return float(np.median(vals))

    fr, wr = read(fetch_csv), read(write_csv)
    f_cal, w_cal = calibration(fr), calibration(wr)
    f_b, n_f = per_launch(fr)
    w_b, _ = per_launch(wr)
    graph = workloads.make_graph(workload)
    cfg = graph.config
    if key == "tp_mfma_bwd":
        algo = mfma_bwd_bytes(cfg, graph.n_atoms, graph.n_edges)
    else:
        algo = algorithmic_bytes(cfg, graph.n_atoms, graph.n_edges)[key]
    traffic = (f_b * copy_kib / f_cal + w_b * copy_kib / w_cal) * 1024
    rec = {"workload": workload, "kernel": key, "kernel_pattern": pattern,
           "kernel_source_digest": kernel_source_digest(),
           "fetch_kib_per_dispatch": f_b, "write_kib_per_dispatch": w_b, "dispatches": n_f,
           "calibration": {"kernel": "stream_kernel<1> (4 GiB read, 4 GiB written)", "fetch_kib": f_cal,
                           "write_kib": w_cal, "fetch_scale": copy_kib / f_cal, "write_scale": copy_kib / w_cal},
           "traffic_bytes_per_launch": traffic, "algorithmic_bytes_per_launch": algo,
           "traffic_over_algorithmic": traffic / algo}
    with open(traffic_record_path(key, workload), "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


# ------------------------------------------------------------------ probes

def pattern_probe(torch, dev, reps=5):
    """The lmax-3 matrix-core backward's tile stream without its arithmetic
    (csrc/stream_probe.hip, pattern_probe): c = a + b over [E][U][32] fp32 on
    the high-order edges, with 128-, 256- and 512-byte rows per wave, at one
    and two workgroups of 8 waves per compute unit.  ms and TB/s per variant."""
    import ctypes

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2504_16068_amd", "libstream_probe.so"))
    lib.pattern_probe.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint, ctypes.c_void_p]
    graph = workloads.make_graph("high_order")
    n, e, u = graph.n_atoms, graph.n_edges, graph.config.U
    a = torch.rand(e * u * 32, device=dev)
    b = torch.rand(e * u * 32, device=dev)
    c = torch.empty_like(a)
    rp = torch.from_numpy(graph.row_ptr).to(dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    nbytes = 3 * e * u * 32 * 4
    names = ["128B rows, 4 tiles", "128B rows, 6 tiles", "256B rows, 2 tiles", "256B rows, 4 tiles",
             "512B rows, 2 tiles"]
    out = {"workload": f"high_order: {e} edges, U={u}, rows of 32 floats per channel", "bytes": nbytes}
    for variant, name in enumerate(names):
        for per_cu in (1, 2):
            def run():
                rc = lib.pattern_probe(variant, n, u, rp.data_ptr(), a.data_ptr(), b.data_ptr(), c.data_ptr(),
                                       cus * per_cu, stream)
                if rc:
                    raise RuntimeError(f"pattern_probe failed ({rc})")
            run()
            torch.cuda.synchronize()
            t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0.record()
            for _ in range(reps):
                run()
            t1.record()
            torch.cuda.synchronize()
            ms = t0.elapsed_time(t1) / reps
            out[f"{name}, {per_cu} workgroup(s) per CU"] = {"ms": ms, "TBps": nbytes / ms / 1e9}
    if not torch.allclose(c[:4096], a[:4096] + b[:4096]):
        raise RuntimeError("pattern_probe wrote wrong sums")
    del a, b, c
    # the direct kernels' traversal at the headline: one workgroup of 16 waves
    # per center copying whole 4.6 KB edge rows (x -> out, no arithmetic)
    lib.center_copy_probe.argtypes = [ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p]
    hg = workloads.make_graph("headline")
    x = torch.rand(hg.n_edges * 64 * 18, device=dev)
    y = torch.empty_like(x)
    hrp = torch.from_numpy(hg.row_ptr).to(dev)
    run = lambda: lib.center_copy_probe(hg.n_atoms, hrp.data_ptr(), x.data_ptr(), y.data_ptr(), stream)
    if run():
        raise RuntimeError("center_copy_probe failed")
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        run()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    if not torch.equal(x, y):
        raise RuntimeError("center_copy_probe copied wrong values")
    cb = 2 * x.numel() * 4
    out["headline per-center copy (16 waves per center, 4.6 KB rows)"] = {"ms": ms, "TBps": cb / ms / 1e9}
    return out


def stream_probes(torch, dev, n_bytes=4 << 30, reps=5):
    """Rates (GB/s of bytes moved) of plain streams over 4 GiB per tensor, outside
    every cache: read only, one read + one write, two reads + one write, each the
    best over a few launch shapes of the committed probe kernels
    (csrc/stream_probe.hip: non-temporal 16-byte accesses)."""
    import ctypes

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2504_16068_amd", "libstream_probe.so"))
    lib.stream_probe.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_uint, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    n_f4 = n_bytes // 16
    a = torch.empty(n_bytes // 4, device=dev).fill_(1.0)
    b = torch.empty_like(a).fill_(2.0)
    c = torch.empty_like(a)
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    stream = torch.cuda.current_stream(dev).cuda_stream
    out = {}
    for pattern, name, tensors in ((0, "read", 1), (1, "read1_write1", 2), (2, "read2_write1", 3)):
        best = None
        for unroll in (1, 2, 4):
            for blocks in (cus * 8, cus * 32, -(-n_f4 // (256 * unroll))):
                def call():
                    rc = lib.stream_probe(pattern, unroll, blocks, a.data_ptr(), b.data_ptr(), c.data_ptr(), n_f4,
                                          stream)
                    if rc != 0:
                        raise RuntimeError(f"stream_probe failed ({rc})")
                call()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(reps):
                    call()
                e1.record()
                torch.cuda.synchronize()
                gbps = tensors * n_bytes / (e0.elapsed_time(e1) / reps / 1e3) / 1e9
                if best is None or gbps > best["GBps"]:
                    best = {"GBps": gbps, "unroll": unroll, "blocks": blocks}
        out[name] = best
    del a, b, c
    torch.cuda.empty_cache()
    return out


# the access pattern of each call, for its probe fraction
PATTERN = {"env_embed": "read", "tp_forward": "read1_write1", "tp_backward": "read2_write1"}


# ------------------------------------------------------------- the step

def time_step(torch, at, dev, name, steps, warmup, with_training=True):
    """Time the hot path (env_embed, tp_forward, tp_backward) on one workload: the
    wall time of `steps` steps between synchronisations, and each call's mean
    duration from HIP events on the library's stream."""
    graph = workloads.make_graph(name)
    cfg = graph.config
    n_atoms, n_edges = graph.n_atoms, graph.n_edges
    if cfg.host_features:
        xh, wh, _, gh = workloads.host_features(cfg, n_edges)
        x, w, g = (torch.from_numpy(a).to(dev) for a in (xh, wh, gh))
    else:
        x, w, g = workloads.device_features(cfg, n_edges, dev)
    pw = torch.from_numpy(workloads.path_weights(cfg)).to(dev)
    rp = torch.from_numpy(graph.row_ptr).to(dev)
    y = torch.from_numpy(graph.Y).to(dev)
    plan = at.allegro_tp_plan_create(cfg.lmax, cfg.U, at.ALLEGRO_FULL_PARITY if cfg.full_parity else 0)
    env = torch.empty((n_atoms, cfg.U, plan.d2), device=dev)
    out = torch.empty_like(x)
    grads = (torch.empty_like(x), torch.empty_like(env), torch.empty_like(w), torch.empty_like(y))

    def step():
        at.allegro_env_embed(plan, rp, w, y, env=env)
        at.allegro_tp_forward(plan, rp, x, env, pw, out=out)
        at.allegro_tp_backward(plan, rp, x, env, pw, g, w, y, outs=grads)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for k in range(steps):
        ev[k][0].record()
        at.allegro_env_embed(plan, rp, w, y, env=env)
        ev[k][1].record()
        at.allegro_tp_forward(plan, rp, x, env, pw, out=out)
        ev[k][2].record()
        at.allegro_tp_backward(plan, rp, x, env, pw, g, w, y, outs=grads)
        ev[k][3].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    names = ("env_embed", "tp_forward", "tp_backward")
    kernel_ms = {nm: float(np.mean([ev[k][i].elapsed_time(ev[k][i + 1]) for k in range(steps)]))
                 for i, nm in enumerate(names)}
    algo = algorithmic_bytes(cfg, n_atoms, n_edges)
    res = {"graph": graph, "cfg": cfg, "plan": plan, "n_atoms": n_atoms, "n_edges": n_edges,
           "ms_per_step": wall * 1e3 / steps, "kernel_ms": kernel_ms,
           "step_event_ms": float(np.mean([ev[k][0].elapsed_time(ev[k][3]) for k in range(steps)])),
           "algo": algo,
           "hbm_algorithmic_GBps": {nm: algo[nm] / (kernel_ms[nm] / 1e3) / 1e9 for nm in names}}
    if with_training:
        res["training_backward"] = time_training_backward(torch, at, plan, (rp, x, env, pw, g, w, y), grads,
                                                          kernel_ms, steps)
    res["tensors"] = (rp, x, env, pw, g, w, y, out, grads)
    return res


def time_training_backward(torch, at, plan, inputs, grads, per_kernel_ms, reps):
    """The training backward (also grad_path_w), timed outside the step: the
    whole call, and the extra time over the inference backward."""
    rp, x, env, pw, g, w, y = inputs
    ws = torch.empty(at.allegro_tp_backward_workspace(plan, rp.numel() - 1), dtype=torch.uint8, device=x.device)
    outs = (*grads, torch.empty_like(pw))

    def call():
        at.allegro_tp_backward_train(plan, rp, x, env, pw, g, w, y, outs=outs, workspace=ws)

    call()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        call()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    del ws
    return {"ms": ms, "extra_over_backward_ms": ms - per_kernel_ms["tp_backward"],
            "workspace_bytes": at.allegro_tp_backward_workspace(plan, rp.numel() - 1)}


def time_harmonics(torch, at, plan, graph, dev, reps):
    """Timings of the fp64 harmonics of the edge vectors and their Cartesian VJP (outside the step).

    Algorithmic bytes per edge: forward reads r (24 B) and writes Y (4 d2 B); the
    backward reads r and grad_Y and writes grad_r (24 B).
    """
    e, d2 = graph.n_edges, plan.d2
    vec = torch.from_numpy(graph.vec).to(dev)
    y = torch.empty((e, d2), device=dev)
    gy = torch.ones((e, d2), device=dev)
    gv = torch.empty((e, 3), device=dev, dtype=torch.float64)
    calls = {"sh_forward": lambda: at.allegro_sh_forward(plan, vec, Y=y),
             "sh_backward": lambda: at.allegro_sh_backward(plan, vec, gy, grad_vec=gv)}
    nbytes = {"sh_forward": e * (24 + 4 * d2), "sh_backward": e * (48 + 4 * d2)}
    res = {}
    for name, fn in calls.items():
        fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / reps
        res[name] = {"ms": ms, "hbm_algorithmic_GBps": nbytes[name] / (ms / 1e3) / 1e9}
    del vec, y, gy, gv
    return res


def roofline(kernel, algo_bytes, ms, probes, traffic):
    achieved = algo_bytes / (ms / 1e3) / 1e9
    probe = probes[PATTERN[kernel]]["GBps"]
    return {"kernel": kernel, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic, "algorithmic_bytes_per_launch": algo_bytes,
            "probe_pattern": PATTERN[kernel], "probe_GBps": probe, "frac_of_probe": achieved / probe}


# ------------------------------------------------------------------- layer

def layer_algorithmic_bytes(cfg, n_edges: int):
    """Least bytes one layer must move: every input read once, every output written once.

    forward:  read h [E,L], V [E,U,d1], Y [E,d2]; write h' [E,L], V' [E,U,d1]
    backward: read h, V, Y, dh' and dV'; write dh, dV, dY
    (weights, row_ptr and the per-center env are under 0.5% and left out; the
    activations the forward saves for the backward are an implementation
    choice and are not counted).
    """
    d1, d2, _ = workloads.dims(cfg.lmax, cfg.full_parity)
    L, UD = cfg.extra["L"], cfg.U * d1
    fwd = 4 * n_edges * (2 * L + 2 * UD + d2)
    bwd = 4 * n_edges * (3 * L + 3 * UD + 2 * d2)
    return {"forward": fwd, "backward": bwd}


def time_layer(torch, at, dev, reps, name="medium_layer"):
    """One Allegro layer (tensor product, mixing, latent MLP, all weight gradients) at the
    medium model shape: forward and backward timed separately with HIP events."""
    graph = workloads.make_graph(name)
    cfg = graph.config
    L, H, e = cfg.extra["L"], cfg.extra["H"], graph.n_edges
    plan = at.allegro_tp_plan_create(cfg.lmax, cfg.U, at.ALLEGRO_FULL_PARITY if cfg.full_parity else 0)
    prm = {k: torch.from_numpy(v).to(dev) for k, v in workloads.layer_params(cfg).items()}
    h, V, dh_out, dV_out = workloads.layer_inputs(cfg, e, dev)
    rp, y = torch.from_numpy(graph.row_ptr).to(dev), torch.from_numpy(graph.Y).to(dev)
    sv_b, ws_b = at.allegro_layer_buffers(plan, L, H, graph.n_atoms, e)
    saved = torch.empty(sv_b, dtype=torch.uint8, device=dev)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=dev)
    h_out, V_out = torch.empty_like(h), torch.empty_like(V)
    outs = {"h": torch.empty_like(h), "V": torch.empty_like(V), "Y": torch.empty_like(y)}
    outs.update({k: torch.empty_like(v) for k, v in prm.items()})

    def fwd():
        at.allegro_layer_forward(plan, L, H, rp, h, V, y, prm, h_out=h_out, V_out=V_out, saved=saved)

    def bwd():
        at.allegro_layer_backward(plan, L, H, rp, h, V, y, prm, saved, dh_out, dV_out, outs=outs, workspace=ws)

    fwd()
    bwd()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps)]
    for k in range(reps):
        ev[k][0].record()
        fwd()
        ev[k][1].record()
        bwd()
        ev[k][2].record()
    torch.cuda.synchronize()
    f_ms = float(np.mean([ev[k][0].elapsed_time(ev[k][1]) for k in range(reps)]))
    b_ms = float(np.mean([ev[k][1].elapsed_time(ev[k][2]) for k in range(reps)]))
    algo = layer_algorithmic_bytes(cfg, e)
    res = {"workload": f"{name}: {graph.n_atoms} atoms, cutoff {cfg.cutoff} A, {e} edges, U={cfg.U}, "
                       f"lmax={cfg.lmax} full parity, latent L={L}, hidden H={H}",
           "forward_ms": f_ms, "backward_ms": b_ms, "edges_per_s": e / ((f_ms + b_ms) / 1e3),
           "algorithmic_bytes": algo,
           "hbm_algorithmic_GBps": {"forward": algo["forward"] / (f_ms / 1e3) / 1e9,
                                    "backward": algo["backward"] / (b_ms / 1e3) / 1e9},
           "saved_bytes": sv_b, "workspace_bytes": ws_b}
    del saved, ws, h_out, V_out, outs, h, V, dh_out, dV_out
    torch.cuda.empty_cache()
    return res


# ------------------------------------------------------------ CPU baseline

_CPU_JOB = {}


def _cpu_range(rng):
    """One share of the oracle's work: env_embed + forward + backward (fp64 NumPy,
    single-threaded BLAS) on the centers [c0, c1) of the sample in _CPU_JOB."""
    from threadpoolctl import threadpool_limits

    from oracle import tp as otp

    c0, c1 = rng
    d = _CPU_JOB
    rp = d["row_ptr"]
    s, e = int(rp[c0]), int(rp[c1])
    if e == s:
        return 0
    local = rp[c0:c1 + 1] - s
    with threadpool_limits(1):
        env = otp.env_embed(local, d["w"][s:e], d["Y"][s:e])
        d["tp"].forward(local, d["x"][s:e], env, d["pw"])
        d["tp"].backward(local, d["x"][s:e], env, d["pw"], d["g"][s:e], d["w"][s:e], d["Y"][s:e])
    return e - s


# (workload, edges of the multi-process sample (None: the whole workload), edges of the single-process sample)
CPU_SAMPLES = (("small", None, 4096), ("headline", 1 << 18, 4096), ("high_order", 1 << 15, 1024))


def cpu_baseline(reps=3):
    """The fp64 oracle (env_embed + forward + backward) timed on the host, before the
    GPU is used: on each workload of CPU_SAMPLES, whole center segments split into
    one range per process over every core of the affinity mask (at most the host
    share of one GPU), and a smaller prefix in a single process; best of `reps`
    time.perf_counter runs each.  The small workload's inputs are the GPU run's own;
    headline and high-order, whose GPU inputs are drawn on the device, use host
    draws of the same distributions."""
    import multiprocessing as mp

    from oracle import tp as otp

    affinity = len(os.sched_getaffinity(0))
    procs = max(1, min(affinity, HOST_SHARE))
    ctx = mp.get_context("fork")  # the GPU is not initialised yet
    per = {}
    for name, multi_edges, single_edges in CPU_SAMPLES:
        graph = workloads.make_graph(name)
        cfg = graph.config
        rp = graph.row_ptr
        n_multi = graph.n_atoms if multi_edges is None else workloads.segment_prefix(rp, multi_edges)
        e_multi = int(rp[n_multi])
        x, w, pw, g = workloads.host_features(cfg, e_multi)
        _CPU_JOB.clear()
        _CPU_JOB.update(row_ptr=rp[:n_multi + 1], x=x, w=w, Y=graph.Y[:e_multi], pw=pw, g=g,
                        tp=otp.TensorProduct(cfg.lmax, cfg.full_parity))
        cuts = [0]
        for k in range(1, procs):
            cuts.append(max(cuts[-1], workloads.segment_prefix(rp[:n_multi + 1], k * e_multi // procs)))
        cuts.append(n_multi)
        ranges = [(a, b) for a, b in zip(cuts[:-1], cuts[1:]) if b > a]
        multi = float("inf")
        with ctx.Pool(procs) as pool:
            for _ in range(reps):
                t0 = time.perf_counter()
                done = sum(pool.map(_cpu_range, ranges, chunksize=1))
                multi = min(multi, time.perf_counter() - t0)
        n_single = workloads.segment_prefix(rp, single_edges)
        e_single = int(rp[n_single])
        single = float("inf")
        for _ in range(reps):
            t0 = time.perf_counter()
            _cpu_range((0, n_single))
            single = min(single, time.perf_counter() - t0)
        per[name] = {"edges_per_s": done / multi, "processes": procs, "sample_edges": done,
                     "sample_centers": n_multi, "seconds": multi,
                     "single_process_edges_per_s": e_single / single, "single_sample_edges": e_single}
        _CPU_JOB.clear()
    head = per["headline"]
    return {"value": head["edges_per_s"], "unit": "edges/s", "cores": procs, "affinity_cores": affinity,
            "kind": "oracle",
            "sample": f"headline: first {head['sample_centers']} centers ({head['sample_edges']} edges) in "
                      f"{procs} ranges of whole segments, one process each (fork, before GPU use): env_embed + "
                      f"forward + backward, fp64 NumPy with single-threaded BLAS, best of {reps}; host-drawn "
                      f"features of the same distributions",
            "per_workload": per}


# -------------------------------------------------------------------- main

def note(msg):
    """A progress line on stderr (stdout carries only the JSON line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="headline", choices=sorted(workloads.CONFIGS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-layer", action="store_true", help="skip the Allegro layer timing")
    ap.add_argument("--no-high-order", action="store_true", help="skip the high-order record")
    ap.add_argument("--no-large", action="store_true", help="skip the large-system record")
    ap.add_argument("--layer-only", action="store_true",
                    help="time only the Allegro layer and print its record (no step, no JSON bench line)")
    ap.add_argument("--pattern-probe", action="store_true",
                    help="time the lmax-3 matrix-core backward's access pattern alone (high-order edges) and exit")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write a calibrated traffic record from two rocprofv3 --pmc runs and exit")
    ap.add_argument("--pmc-kernel", default="tp_backward", choices=sorted(TRAFFIC_KERNELS))
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary, args.workload, args.pmc_kernel)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the tensor product shards by center ranges with no "
              "communication inside the path; each GPU would run this on its own share.", file=sys.stderr)
        sys.exit(2)

    cpu = None if args.no_cpu_baseline or args.layer_only or args.pattern_probe else cpu_baseline()
    if cpu is not None:
        note(f"cpu baseline done: {cpu['value']:.3g} edges/s on {cpu['cores']} processes")

    import torch

    import paper_2504_16068_amd as at

    dev = torch.device("cuda:0")
    if args.layer_only:
        print(json.dumps({"allegro_layer": time_layer(torch, at, dev, max(3, min(args.steps, 10)))}), flush=True)
        return
    if args.pattern_probe:
        print(json.dumps({"pattern_probe": pattern_probe(torch, dev)}), flush=True)
        return
    probes = stream_probes(torch, dev)
    note("stream probes done: " + ", ".join(f"{k} {v['GBps']:.0f} GB/s" for k, v in probes.items()))
    st = time_step(torch, at, dev, args.workload, args.steps, args.warmup)
    note(f"{args.workload} step done: {st['ms_per_step']:.3f} ms")
    cfg, plan, graph = st["cfg"], st["plan"], st["graph"]
    n_atoms, n_edges = st["n_atoms"], st["n_edges"]
    harmonics = time_harmonics(torch, at, plan, graph, dev, args.steps)
    km, algo = st["kernel_ms"], st["algo"]
    result = {
        "metric": METRIC,
        "value": n_edges / (st["ms_per_step"] / 1e3),
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": st["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{args.workload}: {n_atoms} atoms at 0.1/A^3 in a periodic cube, cutoff {cfg.cutoff} A, "
                        f"{n_edges} edges (CSR by center), U={cfg.U}, lmax={cfg.lmax}, "
                        f"{'full' if cfg.full_parity else 'natural'} parity",
            "atoms": n_atoms, "edges": n_edges, "U": cfg.U, "lmax": cfg.lmax,
            "parity": "full" if cfg.full_parity else "natural", "paths": plan.n_paths, "cg_nnz": plan.nnz,
        },
        "kernel_ms": km,
        "step_event_ms": st["step_event_ms"],
        "hbm_algorithmic_GBps": st["hbm_algorithmic_GBps"],
        "frac_of_probe": {nm: st["hbm_algorithmic_GBps"][nm] / probes[PATTERN[nm]]["GBps"] for nm in km},
        "roofline": roofline("tp_backward", algo["tp_backward"], km["tp_backward"], probes,
                             measured_traffic("tp_backward", args.workload)),
        "stream_probes": probes,
        "edge_harmonics": harmonics,
        "training_backward": st["training_backward"],
        "kernel_source_digest": kernel_source_digest(),
    }
    del st
    torch.cuda.empty_cache()
    # the other workloads of the paper's Table I shapes: the large model (lmax 3,
    # 128 channels) and the headline model on a system 5x larger
    for key, skip, steps in (("high_order", args.no_high_order, 10), ("large", args.no_large, 5)):
        if skip or args.workload == key:
            continue
        ot = time_step(torch, at, dev, key, min(args.steps, steps), args.warmup)
        note(f"{key} step done: {ot['ms_per_step']:.3f} ms")
        ok, oa, oc = ot["kernel_ms"], ot["algo"], ot["cfg"]
        result[key] = {
            "workload": f"{key}: {ot['n_atoms']} atoms, cutoff {oc.cutoff} A, {ot['n_edges']} edges, "
                        f"U={oc.U}, lmax={oc.lmax}, {'full' if oc.full_parity else 'natural'} parity",
            "ms_per_step": ot["ms_per_step"], "edges_per_s": ot["n_edges"] / (ot["ms_per_step"] / 1e3),
            "kernel_ms": ok, "hbm_algorithmic_GBps": ot["hbm_algorithmic_GBps"],
            "frac_of_probe": {nm: ot["hbm_algorithmic_GBps"][nm] / probes[PATTERN[nm]]["GBps"] for nm in ok},
            "roofline": roofline("tp_backward", oa["tp_backward"], ok["tp_backward"], probes,
                                 measured_traffic("tp_backward", key)),
            "training_backward": ot["training_backward"]}
        del ot
        torch.cuda.empty_cache()
    if not args.no_layer:
        result["allegro_layer"] = time_layer(torch, at, dev, max(3, min(args.steps, 10)))
        note("layer done")
    if cpu is not None:
        result["cpu_baseline"] = cpu
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
