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
with HIP events on the stream the library launches on.  cpu_baseline times
the fp64 oracle on a prefix of whole center segments, one thread per host core.

The allegro_layer object times one whole Allegro layer (forward, and backward
with every weight gradient) at the medium model shape of Table I, outside the
step.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline] [--no-layer]
       python bench.py --pmc-summary FETCH_CSV WRITE_CSV   (after two rocprofv3 --pmc runs)
"""

from __future__ import annotations

import argparse
import hashlib
import json
import re
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads  # noqa: E402

METRIC = "Allegro TP fwd+bwd edges/sec at lmax=2, 64 ch; % of HBM (or MFMA) roofline"
HBM_PEAK_GBPS = 8000.0
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "tp_backward_headline_traffic.json")


def algorithmic_bytes(cfg, n_atoms: int, n_edges: int):
    """Bytes each kernel must move at least once (fp32 data, int64 row_ptr).

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


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    # every source the tensor-product kernels are compiled from
    for rel in ("paper_2504_16068_amd/csrc/allegro_tp.hip", "paper_2504_16068_amd/csrc/device_common.hpp",
                "paper_2504_16068_amd/csrc/gen_kernels.cpp", "paper_2504_16068_amd/csrc/cg_builder.cpp",
                "paper_2504_16068_amd/csrc/cg_builder.hpp"):
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per tp_backward launch from the committed rocprofv3 counters, if they
    were taken on the current kernel sources and this workload; else None."""
    if not os.path.exists(PROFILE_TRAFFIC):
        return None
    with open(PROFILE_TRAFFIC) as f:
        rec = json.load(f)
    if rec.get("kernel_source_digest") != kernel_source_digest() or rec.get("workload") != workload:
        return None
    return rec.get("traffic_bytes_per_launch")


def pmc_summary(fetch_csv: str, write_csv: str, workload: str, out_path: str):
    """Calibrated HBM traffic of tp_backward from two rocprofv3 --pmc runs of this script.

    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are each scaled by what the same
    counter reads for the 4 GiB device copy that copy_bandwidth() performs
    (__amd_rocclr_copyBuffer), so that request-size conventions of the counters
    cancel out.  Writes the record bench.py reads as roofline.traffic.
    """
    import csv

    def read(path):
        with open(path) as f:
            return list(csv.DictReader(f))

    copy_kib = (4 << 30) / 1024

    def per_launch(rows, kernel):
        # the inference backward only (template arguments: core (lmax, parity),
        # U, the training flag false, then the waves per center), not the
        # training variant
        pat = re.compile(kernel + r"<TPCore<\d+,\s*(true|false)>,\s*\d+,\s*false(,\s*\d+)?>")
        vals = [float(r["Counter_Value"]) for r in rows if pat.search(r["Kernel_Name"])]
        return sum(vals) / len(vals), len(vals)

    fr, wr = read(fetch_csv), read(write_csv)
    f_copy = max(float(r["Counter_Value"]) for r in fr if "copyBuffer" in r["Kernel_Name"])
    w_copy = max(float(r["Counter_Value"]) for r in wr if "copyBuffer" in r["Kernel_Name"])
    f_b, n_f = per_launch(fr, "tp_backward_kernel")
    w_b, _ = per_launch(wr, "tp_backward_kernel")
    graph = workloads.make_graph(workload)
    algo = algorithmic_bytes(graph.config, graph.n_atoms, graph.n_edges)["tp_backward"]
    traffic = (f_b * copy_kib / f_copy + w_b * copy_kib / w_copy) * 1024
    rec = {"workload": workload, "kernel": "tp_backward", "kernel_source_digest": kernel_source_digest(),
           "fetch_kib_per_dispatch": f_b, "write_kib_per_dispatch": w_b, "dispatches": n_f,
           "copy_calibration": {"copy_bytes": 4 << 30, "fetch_kib": f_copy, "write_kib": w_copy,
                                "fetch_scale": copy_kib / f_copy, "write_scale": copy_kib / w_copy},
           "traffic_bytes_per_launch": traffic, "algorithmic_bytes_per_launch": algo,
           "traffic_over_algorithmic": traffic / algo}
    with open(out_path, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def copy_bandwidth(torch, dev, n_bytes=4 << 30, reps=10):
    src = torch.empty(n_bytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    sec = a.elapsed_time(b) / 1e3 / reps
    del src, dst
    torch.cuda.empty_cache()
    return 2 * n_bytes / sec / 1e9


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


def cpu_baseline(graph, host_inputs, edges_per_thread=24576, max_threads=16):
    """Time the fp64 oracle on a prefix of whole center segments of the workload.

    One Python thread per host core (at most max_threads, the host share of one
    GPU), each running env_embed + forward + backward on its own range of
    whole segments with single-threaded BLAS; NumPy releases the GIL inside its
    array loops, so the threads run in parallel.  The single-thread rate on the
    first range is reported beside it.
    """
    from concurrent.futures import ThreadPoolExecutor

    from threadpoolctl import threadpool_limits

    from oracle import tp as otp

    cfg = graph.config
    threads = max(1, min(max_threads, len(os.sched_getaffinity(0))))
    n_end = workloads.segment_prefix(graph.row_ptr, threads * edges_per_thread)
    e_end = int(graph.row_ptr[n_end])
    x, w, pw, g = host_inputs(e_end)
    cuts = [0]
    for k in range(1, threads):
        cuts.append(max(cuts[-1], workloads.segment_prefix(graph.row_ptr, k * edges_per_thread)))
    cuts.append(n_end)
    t = otp.TensorProduct(cfg.lmax, cfg.full_parity)

    def run(k):
        c0, c1 = cuts[k], cuts[k + 1]
        s, e = int(graph.row_ptr[c0]), int(graph.row_ptr[c1])
        if e == s:
            return 0
        rp = graph.row_ptr[c0:c1 + 1] - s
        env = otp.env_embed(rp, w[s:e], graph.Y[s:e])
        t.forward(rp, x[s:e], env, pw)
        t.backward(rp, x[s:e], env, pw, g[s:e], w[s:e], graph.Y[s:e])
        return e - s

    with threadpool_limits(1):
        t0 = time.perf_counter()
        e_single = run(0)
        sec_single = time.perf_counter() - t0
        with ThreadPoolExecutor(threads) as ex:
            t0 = time.perf_counter()
            done = sum(ex.map(run, range(threads)))
            sec = time.perf_counter() - t0
    return {"value": done / sec, "unit": "edges/s", "cores": threads, "kind": "oracle",
            "sample": f"first {n_end} centers ({done} edges) of the same workload in {threads} ranges of whole "
                      f"segments, one Python thread each: env_embed + forward + backward, fp64 NumPy with "
                      f"single-threaded BLAS, {sec:.1f} s wall",
            "single_thread_value": e_single / sec_single,
            "single_thread_sample": f"first {cuts[1]} centers ({e_single} edges), {sec_single:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="headline", choices=sorted(workloads.CONFIGS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-layer", action="store_true", help="skip the Allegro layer timing")
    ap.add_argument("--layer-only", action="store_true",
                    help="time only the Allegro layer and print its record (no step, no JSON bench line)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the calibrated tp_backward traffic record from two rocprofv3 --pmc runs and exit")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary, args.workload, PROFILE_TRAFFIC)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the tensor product shards by center ranges with no "
              "communication inside the path; each GPU would run this on its own share.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2504_16068_amd as at

    dev = torch.device("cuda:0")
    if args.layer_only:
        print(json.dumps({"allegro_layer": time_layer(torch, at, dev, max(3, min(args.steps, 10)))}), flush=True)
        return
    graph = workloads.make_graph(args.workload)
    cfg = graph.config
    n_atoms, n_edges = graph.n_atoms, graph.n_edges
    if cfg.host_features:
        xh, wh, pwh, gh = workloads.host_features(cfg, n_edges)
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

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for k in range(args.steps):
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
    per_kernel_ms = {nm: float(np.mean([ev[k][i].elapsed_time(ev[k][i + 1]) for k in range(args.steps)]))
                     for i, nm in enumerate(names)}
    ms_per_step = wall * 1e3 / args.steps
    value = n_edges / (ms_per_step / 1e3)

    harmonics = time_harmonics(torch, at, plan, graph, dev, args.steps)
    training = time_training_backward(torch, at, plan, (rp, x, env, pw, g, w, y), grads, per_kernel_ms, args.steps)
    algo = algorithmic_bytes(cfg, n_atoms, n_edges)
    bwd_s = per_kernel_ms["tp_backward"] / 1e3
    achieved = algo["tp_backward"] / bwd_s / 1e9
    copy_gbps = copy_bandwidth(torch, dev)
    traffic = measured_traffic(args.workload)

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
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
        "kernel_ms": per_kernel_ms,
        "step_event_ms": float(np.mean([ev[k][0].elapsed_time(ev[k][3]) for k in range(args.steps)])),
        "hbm_algorithmic_GBps": {nm: algo[nm] / (per_kernel_ms[nm] / 1e3) / 1e9 for nm in names},
        "copy_GBps_measured": copy_gbps,
        "roofline": {
            "kernel": "tp_backward",
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": algo["tp_backward"],
            "frac_of_measured_copy": achieved / copy_gbps,
        },
        "edge_harmonics": harmonics,
        "training_backward": training,
        "kernel_source_digest": kernel_source_digest(),
    }
    del x, w, g, out, grads, env
    torch.cuda.empty_cache()
    if not args.no_layer:
        result["allegro_layer"] = time_layer(torch, at, dev, max(3, min(args.steps, 10)))
    if not args.no_cpu_baseline:
        cfg_ = cfg

        def host_inputs(e):
            if cfg_.host_features:
                return xh[:e], wh[:e], pwh, gh[:e]
            xs, ws, gs = workloads.device_features(cfg_, n_edges, dev)
            res = xs[:e].cpu().numpy(), ws[:e].cpu().numpy(), workloads.path_weights(cfg_), gs[:e].cpu().numpy()
            del xs, ws, gs
            torch.cuda.empty_cache()
            return res

        result["cpu_baseline"] = cpu_baseline(graph, host_inputs)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
