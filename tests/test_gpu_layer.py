"""GPU parity of one Allegro layer (include/allegro_layer.h) against the fp64 oracle.

The layer composes the tensor product with dense fp32 contractions on the
matrix cores (environment weights, per-irrep channel mixing, the latent MLP)
and their VJPs, including every weight gradient.  Small inputs are compared
element by element.  At the medium model shape (about 1e6 edges, lmax 3, 64
channels) the per-edge outputs are compared on sampled center segments,
which the oracle evaluates from the segments' own inputs; the weight
gradients, which sum over every edge, are checked by additivity over ranges
of centers (the full run against the sum of the runs on the ranges) and one
range against the oracle.
"""

import sys

import numpy as np
import pytest

import workloads
from oracle import layer as olayer
from tests.parity import BWD_TOL, FWD_TOL, block_rel_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

DEV = "cuda:0"
WEIGHTS = ("A", "W", "Mix", "B1", "B2")


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def at():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    import paper_2504_16068_amd as lib
    return lib


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _plan(at, lmax, full):
    return at.allegro_tp_plan_create(lmax, 64, at.ALLEGRO_FULL_PARITY if full else 0)


def _gpu_layer(at, plan, L, H, row_ptr, h, V, Y, prm, dh_out, dV_out):
    """Forward and backward through the C ABI; returns numpy (h_out, V_out, grads)."""
    rp, hd, Vd, Yd, dhd, dVd = (a if isinstance(a, torch.Tensor) else _t(a) for a in (row_ptr, h, V, Y, dh_out, dV_out))
    wd = {k: (v if isinstance(v, torch.Tensor) else _t(v)) for k, v in prm.items()}
    h_out, V_out, saved = at.allegro_layer_forward(plan, L, H, rp, hd, Vd, Yd, wd)
    grads = at.allegro_layer_backward(plan, L, H, rp, hd, Vd, Yd, wd, saved, dhd, dVd)
    torch.cuda.synchronize()
    return h_out, V_out, grads


def _np(t):
    return t.cpu().numpy()


def _compare(lay, got, ref, tag, weight_grads=True):
    (h_o, V_o, g), (rh_o, rV_o, rg) = got, ref
    xs = lay.tp.x_slices
    errs = {"h_out": (block_rel_err(h_o, rh_o), FWD_TOL), "V_out": (block_rel_err(V_o, rV_o, xs), FWD_TOL),
            "dh": (block_rel_err(g["h"], rg["h"]), BWD_TOL), "dV": (block_rel_err(g["V"], rg["V"], xs), BWD_TOL),
            "dY": (block_rel_err(g["Y"], rg["Y"], lay.tp.env_slices), BWD_TOL)}
    if weight_grads:
        for k in WEIGHTS:
            errs["d" + k] = (block_rel_err(g[k], rg[k]), BWD_TOL)
    _note(f"{tag}: " + ", ".join(f"{k}={v:.2e}" for k, (v, _) in errs.items()))
    bad = {k: v for k, (v, tol) in errs.items() if not v <= tol}
    assert not bad, f"{tag}: parity failed {bad}"


def _oracle(lmax, full, L, H, row_ptr, h, V, Y, prm, dh_out, dV_out):
    lay = olayer.AllegroLayer(lmax, full, 64, L, H)
    h_o, V_o, _ = lay.forward(row_ptr, h, V, Y, prm)
    return lay, (h_o, V_o, lay.backward(row_ptr, h, V, Y, prm, dh_out, dV_out))


def _host(t):
    return {k: (_np(v) if isinstance(v, torch.Tensor) else v) for k, v in t.items()}


def test_layer_small_workload(at):
    graph = workloads.make_graph("layer_small")
    cfg = graph.config
    L, H = cfg.extra["L"], cfg.extra["H"]
    prm = workloads.layer_params(cfg)
    h, V, dh_out, dV_out = workloads.layer_inputs(cfg, graph.n_edges)
    _note(f"[gpu] layer_small: N={graph.n_atoms} E={graph.n_edges} lmax={cfg.lmax} L={L} H={H}")
    plan = _plan(at, cfg.lmax, cfg.full_parity)
    h_o, V_o, g = _gpu_layer(at, plan, L, H, graph.row_ptr, h, V, graph.Y, prm, dh_out, dV_out)
    lay, ref = _oracle(cfg.lmax, cfg.full_parity, L, H, graph.row_ptr, h, V, graph.Y, prm, dh_out, dV_out)
    _compare(lay, (_np(h_o), _np(V_o), _host(g)), ref, "layer_small")


def test_two_stacked_layers(at):
    """Two layers in sequence on layer_small (the paper's model stacks layers, each
    taking the previous one's (h, V) and the same edge harmonics Y, Table I):
    the second layer's output and, through both backwards chained on the device,
    the input gradients, dY (summed over both layers) and every weight gradient
    of both layers against the oracle chained in fp64."""
    import dataclasses

    graph = workloads.make_graph("layer_small")
    cfg = graph.config
    L, H = cfg.extra["L"], cfg.extra["H"]
    prm1 = workloads.layer_params(cfg)
    prm2 = workloads.layer_params(dataclasses.replace(cfg, index=cfg.index + 1000))
    h, V, dh_out, dV_out = workloads.layer_inputs(cfg, graph.n_edges)
    _note(f"[gpu] two stacked layers on layer_small: N={graph.n_atoms} E={graph.n_edges}")
    plan = _plan(at, cfg.lmax, cfg.full_parity)
    rp, Yd = _t(graph.row_ptr), _t(graph.Y)
    w1, w2 = ({k: _t(v) for k, v in p.items()} for p in (prm1, prm2))
    h1, V1, saved1 = at.allegro_layer_forward(plan, L, H, rp, _t(h), _t(V), Yd, w1)
    h2, V2, saved2 = at.allegro_layer_forward(plan, L, H, rp, h1, V1, Yd, w2)
    g2 = at.allegro_layer_backward(plan, L, H, rp, h1, V1, Yd, w2, saved2, _t(dh_out), _t(dV_out))
    g1 = at.allegro_layer_backward(plan, L, H, rp, _t(h), _t(V), Yd, w1, saved1, g2["h"], g2["V"])
    torch.cuda.synchronize()

    lay = olayer.AllegroLayer(cfg.lmax, cfg.full_parity, 64, L, H)
    rh1, rV1, _ = lay.forward(graph.row_ptr, h, V, graph.Y, prm1)
    rh2, rV2, _ = lay.forward(graph.row_ptr, rh1, rV1, graph.Y, prm2)
    rg2 = lay.backward(graph.row_ptr, rh1, rV1, graph.Y, prm2, dh_out, dV_out)
    rg1 = lay.backward(graph.row_ptr, h, V, graph.Y, prm1, rg2["h"], rg2["V"])
    xs = lay.tp.x_slices
    errs = {"h_out": (block_rel_err(_np(h2), rh2), FWD_TOL), "V_out": (block_rel_err(_np(V2), rV2, xs), FWD_TOL),
            "dh": (block_rel_err(_np(g1["h"]), rg1["h"]), BWD_TOL),
            "dV": (block_rel_err(_np(g1["V"]), rg1["V"], xs), BWD_TOL),
            "dY": (block_rel_err(_np(g1["Y"]) + _np(g2["Y"]), rg1["Y"] + rg2["Y"], lay.tp.env_slices), BWD_TOL)}
    for k in WEIGHTS:
        errs["d" + k + "1"] = (block_rel_err(_np(g1[k]), rg1[k]), BWD_TOL)
        errs["d" + k + "2"] = (block_rel_err(_np(g2[k]), rg2[k]), BWD_TOL)
    _note("two layers: " + ", ".join(f"{k}={v:.2e}" for k, (v, _) in errs.items()))
    bad = {k: v for k, (v, tol) in errs.items() if not v <= tol}
    assert not bad, f"two layers: parity failed {bad}"


def _synthetic(lmax, full, L, H, degrees, seed):
    rng = np.random.default_rng(seed)
    degrees = np.asarray(degrees, dtype=np.int64)
    row_ptr = np.concatenate([[0], np.cumsum(degrees)]).astype(np.int64)
    e = int(row_ptr[-1])
    d1, d2, n_paths = workloads.dims(lmax, full)
    n_x = 2 * (lmax + 1) if full else lmax + 1
    vec = rng.standard_normal((max(e, 1), 3))[:e]
    Y = workloads.real_sh_cartesian(lmax, vec).astype(np.float32) if e else np.zeros((0, d2), np.float32)
    f32 = np.float32
    h = rng.standard_normal((e, L), dtype=f32)
    V = rng.standard_normal((e, 64, d1), dtype=f32)
    prm = {"A": rng.standard_normal((L, 64), dtype=f32) / f32(np.sqrt(L)),
           "W": rng.standard_normal((n_paths, 64), dtype=f32) / f32(np.sqrt(n_paths)),
           "Mix": rng.standard_normal((n_x, 64, 64), dtype=f32) / f32(8.0),
           "B1": rng.standard_normal((L + 64, H), dtype=f32) / f32(np.sqrt(L + 64)),
           "B2": rng.standard_normal((H, L), dtype=f32) / f32(np.sqrt(H))}
    dh_out = rng.standard_normal((e, L), dtype=f32)
    dV_out = rng.standard_normal((e, 64, d1), dtype=f32)
    return row_ptr, h, V, Y, prm, dh_out, dV_out


LAYER_CASES = [
    # (lmax, full, L, H, degrees): empty segments and edge counts that leave ragged
    # tails in every tile size (64-row GEMM tiles, 8- and 4-edge mixing tiles)
    (1, False, 64, 64, [0, 3, 0, 17, 1]),
    (1, True, 128, 64, [5, 0, 66, 2]),
    (2, True, 64, 128, [0, 1, 2, 63, 64, 65, 0]),
    (2, False, 128, 128, [31, 0, 9]),
    (3, True, 64, 128, [1, 0, 70, 3]),
    (3, False, 64, 64, [129, 2]),
]


@pytest.mark.parametrize("lmax,full,L,H,degrees", LAYER_CASES)
def test_layer_edge_cases(at, lmax, full, L, H, degrees):
    _note(f"[gpu] layer edge case lmax={lmax} full={full} L={L} H={H} degrees={degrees}")
    data = _synthetic(lmax, full, L, H, degrees, seed=lmax * 1000 + L + H + len(degrees))
    plan = _plan(at, lmax, full)
    h_o, V_o, g = _gpu_layer(at, plan, L, H, *data)
    lay, ref = _oracle(lmax, full, L, H, *data)
    _compare(lay, (_np(h_o), _np(V_o), _host(g)), ref, f"layer lmax{lmax}{'F' if full else 'N'} L{L} H{H}")


def test_layer_without_edges(at):
    """E = 0 with N = 3 centers: empty outputs and zero weight gradients (outputs pre-filled with garbage)."""
    _note("[gpu] layer with E = 0, N = 3")
    lmax, full, L, H = 2, True, 64, 128
    row_ptr, h, V, Y, prm, dh_out, dV_out = _synthetic(lmax, full, L, H, [0, 0, 0], seed=5)
    plan = _plan(at, lmax, full)
    wd = {k: _t(v) for k, v in prm.items()}
    rp, hd, Vd, Yd = _t(row_ptr), _t(h), _t(V), _t(Y)
    h_out, V_out, saved = at.allegro_layer_forward(plan, L, H, rp, hd, Vd, Yd, wd)
    outs = {"h": torch.empty_like(hd), "V": torch.empty_like(Vd), "Y": torch.empty_like(Yd)}
    outs.update({k: torch.full_like(v, 7.0) for k, v in wd.items()})
    g = at.allegro_layer_backward(plan, L, H, rp, hd, Vd, Yd, wd, saved, _t(dh_out), _t(dV_out), outs=outs)
    torch.cuda.synchronize()
    assert h_out.shape == (0, L) and V_out.shape == (0, 64, plan.d1)
    for k in WEIGHTS:
        assert torch.count_nonzero(g[k]).item() == 0, k


def test_layer_run_to_run_identical(at):
    graph = workloads.make_graph("layer_small")
    cfg = graph.config
    L, H = cfg.extra["L"], cfg.extra["H"]
    prm = workloads.layer_params(cfg)
    h, V, dh_out, dV_out = workloads.layer_inputs(cfg, graph.n_edges)
    _note("[gpu] layer run-to-run identity")
    plan = _plan(at, cfg.lmax, cfg.full_parity)
    a = _gpu_layer(at, plan, L, H, graph.row_ptr, h, V, graph.Y, prm, dh_out, dV_out)
    b = _gpu_layer(at, plan, L, H, graph.row_ptr, h, V, graph.Y, prm, dh_out, dV_out)
    for x, y in [(a[0], b[0]), (a[1], b[1])] + [(a[2][k], b[2][k]) for k in a[2]]:
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))


def test_layer_rejects_small_buffers(at):
    lmax, full, L, H = 1, False, 64, 64
    row_ptr, h, V, Y, prm, dh_out, dV_out = _synthetic(lmax, full, L, H, [2, 3], seed=1)
    plan = _plan(at, lmax, full)
    wd = {k: _t(v) for k, v in prm.items()}
    rp, hd, Vd, Yd = _t(row_ptr), _t(h), _t(V), _t(Y)
    sv, ws = at.allegro_layer_buffers(plan, L, H, 2, 5)
    with pytest.raises(at.AllegroError) as ex:
        at.allegro_layer_forward(plan, L, H, rp, hd, Vd, Yd, wd,
                                 saved=torch.empty(sv - 256, dtype=torch.uint8, device=DEV))
    assert ex.value.code == at.ALLEGRO_E_INVALID and "saved" in str(ex.value)
    _, _, saved = at.allegro_layer_forward(plan, L, H, rp, hd, Vd, Yd, wd)
    with pytest.raises(at.AllegroError) as ex:
        at.allegro_layer_backward(plan, L, H, rp, hd, Vd, Yd, wd, saved, _t(dh_out), _t(dV_out),
                                  workspace=torch.empty(ws - 256, dtype=torch.uint8, device=DEV))
    assert ex.value.code == at.ALLEGRO_E_INVALID and "workspace" in str(ex.value)
    torch.cuda.synchronize()


# ------------------------------------------- medium model shape, full size

def _rebased(row_ptr, c0, c1):
    return (row_ptr[c0:c1 + 1] - row_ptr[c0]).astype(np.int64)


def test_layer_medium_full_size(at, n_samples=12, n_ranges=4):
    graph = workloads.make_graph("medium_layer")
    cfg = graph.config
    L, H = cfg.extra["L"], cfg.extra["H"]
    n, e = graph.n_atoms, graph.n_edges
    _note(f"[gpu] medium layer: N={n} E={e} lmax={cfg.lmax} U={cfg.U} L={L} H={H} (sampled)")
    prm = workloads.layer_params(cfg)
    plan = _plan(at, cfg.lmax, cfg.full_parity)
    h, V, dh_out, dV_out = workloads.layer_inputs(cfg, e, DEV)
    rp, Yd = _t(graph.row_ptr), _t(graph.Y)
    wd = {k: _t(v) for k, v in prm.items()}
    h_o, V_o, g = _gpu_layer(at, plan, L, H, rp, h, V, Yd, wd, dh_out, dV_out)

    # per-edge outputs on sampled center segments against the oracle
    rng = np.random.default_rng(cfg.index + 90)
    centers = np.unique(np.concatenate([[0, n - 1], rng.integers(0, n, n_samples)]))
    segs = [(int(graph.row_ptr[c]), int(graph.row_ptr[c + 1])) for c in centers]
    idx_np = np.concatenate([np.arange(s, t) for s, t in segs])
    idx = torch.as_tensor(idx_np, device=DEV)
    local = np.concatenate([[0], np.cumsum([t - s for s, t in segs])]).astype(np.int64)
    sub = [_np(a[idx]) for a in (h, V, dh_out, dV_out)]
    lay, (rh, rV, rg) = _oracle(cfg.lmax, cfg.full_parity, L, H, local, sub[0], sub[1], graph.Y[idx_np], prm,
                                sub[2], sub[3])
    got = (_np(h_o[idx]), _np(V_o[idx]), {k: _np(g[k][idx]) for k in ("h", "V", "Y")})
    _compare(lay, got, (rh, rV, rg), f"medium_layer[{len(centers)} segments]", weight_grads=False)
    del h_o, V_o

    # weight gradients: additivity over center ranges, and one range against the oracle
    bounds = np.linspace(0, n, n_ranges + 1).astype(np.int64)
    total = {k: np.zeros(prm[k].shape) for k in WEIGHTS}
    for r in range(n_ranges):
        c0, c1 = int(bounds[r]), int(bounds[r + 1])
        s, t = int(graph.row_ptr[c0]), int(graph.row_ptr[c1])
        part = [a[s:t].contiguous() for a in (h, V, dh_out, dV_out)]
        _, _, gr = _gpu_layer(at, plan, L, H, _t(_rebased(graph.row_ptr, c0, c1)), part[0], part[1],
                              Yd[s:t].contiguous(), wd, part[2], part[3])
        for k in WEIGHTS:
            total[k] += _np(gr[k]).astype(np.float64)
        del gr, part
    for k in WEIGHTS:
        err = block_rel_err(_np(g[k]), total[k])
        _note(f"medium_layer d{k}: full run vs sum over {n_ranges} center ranges err={err:.2e}")
        assert err <= BWD_TOL, k
    del g
    torch.cuda.empty_cache()
    # a range of whole segments small enough for the oracle (about 3000 edges)
    c1 = workloads.segment_prefix(graph.row_ptr, 3000)
    t = int(graph.row_ptr[c1])
    part = [a[:t].contiguous() for a in (h, V, dh_out, dV_out)]
    hr, Vr, gr = _gpu_layer(at, plan, L, H, _t(graph.row_ptr[:c1 + 1]), part[0], part[1], Yd[:t].contiguous(), wd,
                            part[2], part[3])
    host = [_np(a) for a in part]
    lay, ref = _oracle(cfg.lmax, cfg.full_parity, L, H, graph.row_ptr[:c1 + 1], host[0], host[1], graph.Y[:t], prm,
                       host[2], host[3])
    _compare(lay, (_np(hr), _np(Vr), _host(gr)), ref, f"medium_layer[first {c1} centers, {t} edges]")


def test_layer_replays_in_a_hip_graph(at):
    """Forward and backward of one layer captured once into a HIP graph and replayed
    several times, with eager work and synchronisation between replays; every replay
    must equal the eager result bit for bit."""
    graph = workloads.make_graph("layer_small")
    cfg = graph.config
    L, H = cfg.extra["L"], cfg.extra["H"]
    _note("[gpu] HIP graph replay of one layer, layer_small")
    plan = _plan(at, cfg.lmax, cfg.full_parity)
    prm = {k: _t(v) for k, v in workloads.layer_params(cfg).items()}
    h, V, dh_out, dV_out = (_t(a) for a in workloads.layer_inputs(cfg, graph.n_edges))
    rp, Y = _t(graph.row_ptr), _t(graph.Y)
    sv, ws = at.allegro_layer_buffers(plan, L, H, graph.n_atoms, graph.n_edges)
    saved = torch.empty(sv, dtype=torch.uint8, device=DEV)
    work = torch.empty(ws, dtype=torch.uint8, device=DEV)
    h_out, V_out = torch.empty_like(h), torch.empty_like(V)
    outs = {"h": torch.empty_like(h), "V": torch.empty_like(V), "Y": torch.empty_like(Y)}
    outs.update({k: torch.empty_like(v) for k, v in prm.items()})

    def step():
        at.allegro_layer_forward(plan, L, H, rp, h, V, Y, prm, h_out=h_out, V_out=V_out, saved=saved)
        at.allegro_layer_backward(plan, L, H, rp, h, V, Y, prm, saved, dh_out, dV_out, outs=outs, workspace=work)

    results = [h_out, V_out] + [outs[k] for k in sorted(outs)]
    step()
    torch.cuda.synchronize()
    eager = [r.clone() for r in results]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    hip_graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(hip_graph):
        step()
    for rep in range(3):
        for r in results:
            r.fill_(float("nan"))  # eager work between replays
        saved.fill_(0xFF)
        work.fill_(0xFF)
        torch.cuda.synchronize()
        hip_graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(results, eager):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), rep
