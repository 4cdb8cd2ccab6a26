"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Both sides run the whole pipeline (embedding -> forward -> backward) from the
same seeded fp32 inputs.  Small workloads are compared element by element;
the full-size workloads (about 1e6 and 9e6 edges), run in exactly the launch
configuration the bench times, are compared on sampled center segments, which
the oracle evaluates one by one from the segments' own inputs.
"""

import sys

import numpy as np
import pytest

import workloads
from oracle import tp as otp
from tests.parity import BWD_TOL, FWD_TOL, block_rel_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def at():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    import paper_2504_16068_amd as lib
    return lib


DEV = "cuda:0"


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _plan(at, lmax, U, full, det=False, validate=False):
    flags = (at.ALLEGRO_FULL_PARITY if full else 0) | (at.ALLEGRO_DETERMINISTIC if det else 0)
    flags |= at.ALLEGRO_VALIDATE if validate else 0
    return at.allegro_tp_plan_create(lmax, U, flags)


def _run_gpu(at, plan, row_ptr, x, w, y, pw, g):
    rp, xd, wd, yd, pwd, gd = (_t(a) if isinstance(a, np.ndarray) else a for a in (row_ptr, x, w, y, pw, g))
    env = at.allegro_env_embed(plan, rp, wd, yd)
    out = at.allegro_tp_forward(plan, rp, xd, env, pwd)
    grads = at.allegro_tp_backward(plan, rp, xd, env, pwd, gd, wd, yd)
    torch.cuda.synchronize()
    return env, out, grads


def _oracle(lmax, full, row_ptr, x, w, y, pw, g):
    t = otp.TensorProduct(lmax, full)
    env = otp.env_embed(row_ptr, w, y)
    out = t.forward(row_ptr, x, env, pw)
    return t, env, out, t.backward(row_ptr, x, env, pw, g, w, y)


def _compare(t, gpu, ref, tag):
    env, out, (gx, genv, gw, gy) = gpu
    renv, rout, (rgx, rgenv, rgw, rgy) = ref
    errs = {
        "env": (block_rel_err(env, renv, t.env_slices), FWD_TOL),
        "out": (block_rel_err(out, rout, t.x_slices), FWD_TOL),
        "grad_x": (block_rel_err(gx, rgx, t.x_slices), BWD_TOL),
        "grad_env": (block_rel_err(genv, rgenv, t.env_slices), BWD_TOL),
        "grad_w": (block_rel_err(gw, rgw), BWD_TOL),
        "grad_Y": (block_rel_err(gy, rgy, t.env_slices), BWD_TOL),
    }
    plain = {k: _max_rel(g, o) for k, g, o in (("env", env, renv), ("out", out, rout), ("grad_x", gx, rgx),
                                                ("grad_env", genv, rgenv), ("grad_w", gw, rgw), ("grad_Y", gy, rgy))}
    _note(f"{tag}: " + ", ".join(f"{k}={v:.2e}" for k, (v, _) in errs.items())
          + " | max|g-o|/max|o|: " + ", ".join(f"{k}={v:.2e}" for k, v in plain.items()))
    bad = {k: v for k, (v, tol) in errs.items() if not v <= tol}
    assert not bad, f"{tag}: parity failed {bad}"


def _max_rel(got, ref):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-300)) if ref.size else 0.0


def _np(gpu):
    env, out, grads = gpu
    return env.cpu().numpy(), out.cpu().numpy(), tuple(a.cpu().numpy() for a in grads)


# ------------------------------------------------------------ whole workloads

@pytest.mark.parametrize("name", ["tiny", "small"])
def test_workload_full_parity(at, name):
    graph = workloads.make_graph(name)
    cfg = graph.config
    x, w, pw, g = workloads.host_features(cfg, graph.n_edges)
    _note(f"[gpu] {name}: N={graph.n_atoms} E={graph.n_edges} U={cfg.U} lmax={cfg.lmax}")
    plan = _plan(at, cfg.lmax, cfg.U, cfg.full_parity)
    gpu = _np(_run_gpu(at, plan, graph.row_ptr, x, w, graph.Y, pw, g))
    t, *ref = _oracle(cfg.lmax, cfg.full_parity, graph.row_ptr, x, w, graph.Y, pw, g)
    _compare(t, gpu, ref, name)


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_deterministic_env_is_bit_exact(at, name):
    graph = workloads.make_graph(name)
    cfg = graph.config
    _, w, _, _ = workloads.host_features(cfg, graph.n_edges)
    _note(f"[gpu] deterministic env {name}")
    plan = _plan(at, cfg.lmax, cfg.U, cfg.full_parity, det=True)
    rp, wd, yd = _t(graph.row_ptr), _t(w), _t(graph.Y)
    env1 = at.allegro_env_embed(plan, rp, wd, yd).cpu().numpy()
    env2 = at.allegro_env_embed(plan, rp, wd, yd).cpu().numpy()
    ref = otp.env_embed_fp32_replay(graph.row_ptr, w, graph.Y)
    assert np.array_equal(env1.view(np.uint32), ref.view(np.uint32))
    assert np.array_equal(env1.view(np.uint32), env2.view(np.uint32))


def test_run_to_run_bitwise_identical(at):
    graph = workloads.make_graph("small")
    cfg = graph.config
    x, w, pw, g = workloads.host_features(cfg, graph.n_edges)
    _note("[gpu] run-to-run identity, small")
    plan = _plan(at, cfg.lmax, cfg.U, cfg.full_parity)
    a = _np(_run_gpu(at, plan, graph.row_ptr, x, w, graph.Y, pw, g))
    b = _np(_run_gpu(at, plan, graph.row_ptr, x, w, graph.Y, pw, g))
    for u, v in zip((a[0], a[1], *a[2]), (b[0], b[1], *b[2])):
        assert np.array_equal(u.view(np.uint32), v.view(np.uint32))


# ------------------------------------------------------- synthetic edge cases

def _synthetic(lmax, full, U, degrees, seed):
    rng = np.random.default_rng(seed)
    degrees = np.asarray(degrees, dtype=np.int64)
    row_ptr = np.concatenate([[0], np.cumsum(degrees)]).astype(np.int64)
    n_edges = int(row_ptr[-1])
    d1, d2, n_paths = workloads.dims(lmax, full)
    vec = rng.standard_normal((max(n_edges, 1), 3))[:n_edges]
    y = workloads.real_sh_cartesian(lmax, vec).astype(np.float32) if n_edges else np.zeros((0, d2), np.float32)
    x = rng.standard_normal((n_edges, U, d1), dtype=np.float32)
    w = rng.standard_normal((n_edges, U), dtype=np.float32)
    pw = (rng.standard_normal((n_paths, U)) / np.sqrt(n_paths)).astype(np.float32)
    g = rng.standard_normal((n_edges, U, d1), dtype=np.float32)
    return row_ptr, x, w, y, pw, g


EDGE_CASES = [
    # (lmax, full, U, degrees): empty segments, ragged tails, degree 1, long segments
    (1, False, 16, [0, 1, 0, 5, 17, 0, 3]),
    (1, True, 32, [2, 0, 0, 65, 1]),
    (2, True, 64, [0, 1, 2, 63, 64, 65, 130, 0]),
    (2, False, 128, [7, 0, 33]),
    (3, True, 64, [1, 0, 9, 70]),
    (3, True, 128, [0, 3, 40]),
    (3, False, 16, [5, 6, 0, 1]),
    (2, True, 32, [300]),
]


@pytest.mark.parametrize("lmax,full,U,degrees", EDGE_CASES)
def test_edge_cases(at, lmax, full, U, degrees):
    _note(f"[gpu] edge case lmax={lmax} full={full} U={U} degrees={degrees}")
    data = _synthetic(lmax, full, U, degrees, seed=lmax * 100 + U + len(degrees))
    plan = _plan(at, lmax, U, full, validate=True)
    gpu = _np(_run_gpu(at, plan, *data))
    t, *ref = _oracle(lmax, full, *data)
    _compare(t, gpu, ref, f"lmax{lmax}{'F' if full else 'N'}U{U}")
    env = gpu[0]
    assert np.all(env[np.asarray(degrees) == 0] == 0)


@pytest.mark.parametrize("U", [64, 128])
def test_matrix_forward_tile_boundaries(at, U):
    """The lmax-3 full-parity forward loads 4-edge tiles straight into LDS through
    a ring of four buffers: segment lengths on every side of a tile boundary (0 to
    5, 7 to 9, 12 and 13, 16 and 17, 20 and 21), a ring that wraps several times
    (33, 64, 65 edges), and the backward on the same data, against the oracle."""
    degrees = [0, 1, 2, 3, 4, 5, 7, 8, 9, 12, 13, 16, 17, 20, 21, 33, 64, 65, 0]
    _note(f"[gpu] matrix forward tile boundaries U={U}")
    data = _synthetic(3, True, U, degrees, seed=4242 + U)
    plan = _plan(at, 3, U, True)
    gpu = _np(_run_gpu(at, plan, *data))
    t, *ref = _oracle(3, True, *data)
    _compare(t, gpu, ref, f"lmax3F U{U} tile boundaries")


ALL_SHAPES = [(lmax, full, U) for lmax in (1, 2, 3) for full in (False, True) for U in (16, 32, 64, 128)]


@pytest.mark.parametrize("lmax,full,U", ALL_SHAPES)
def test_every_core_and_width(at, lmax, full, U):
    """Every compiled (lmax, parity) core at every channel count, through the
    embedding, the forward, the inference backward and the training backward,
    on ragged segments (empty, one edge, a partial lane-group pass, more than
    one slab), against the oracle."""
    degrees = [0, 1, 3, 17, 66]
    _note(f"[gpu] shape sweep lmax={lmax} full={full} U={U}")
    data = _synthetic(lmax, full, U, degrees, seed=1000 + lmax * 100 + U + int(full))
    plan = _plan(at, lmax, U, full)
    gpu = _np(_run_gpu(at, plan, *data))
    t, *ref = _oracle(lmax, full, *data)
    _compare(t, gpu, ref, f"sweep lmax{lmax}{'F' if full else 'N'}U{U}")
    rp, xd, wd, yd, pwd, gd = (_t(a) for a in data)
    env = at.allegro_env_embed(plan, rp, wd, yd)
    (gx, genv, gw, gy, gpw), _ = _train(at, plan, rp, xd, env, pwd, gd, wd, yd)
    renv = otp.env_embed(data[0], data[2], data[3])
    rgrads = t.backward(data[0], data[1], renv, data[4], data[5], data[2], data[3])
    for got, r, blocks in zip((gx, genv, gw, gy), rgrads, (t.x_slices, t.env_slices, None, t.env_slices)):
        assert block_rel_err(got.cpu().numpy(), r, blocks) <= BWD_TOL
    err = block_rel_err(gpw.cpu().numpy(), t.path_weight_grad(data[0], data[1], renv, data[5]))
    _note(f"sweep lmax{lmax}{'F' if full else 'N'}U{U}: training grads within {BWD_TOL}, grad_path_w err={err:.2e}")
    assert err <= BWD_TOL


@pytest.mark.parametrize("lmax,full,U", [(2, True, 64), (3, True, 128), (1, False, 16)])
def test_skewed_degrees(at, lmax, full, U):
    """Heavy-tailed segment lengths: many empty centers, many short ones, a few with
    hundreds of edges and one with thousands, so that every wave of a center's
    workgroup gets many slabs, few or none.

    A segment sum over n edges in fp32 carries a rounding error that grows with n,
    so at thousands of edges the relative bars (set for the workloads' ~50
    neighbours) do not apply to env itself.  What is exact or bounded is checked:
    the deterministic env equals the fp32 sequential replay bit for bit; the fast
    env is within the recursive-summation bound gamma_n * sum |w Y| of the fp64
    sum (one rounding per step with FMA, u = 2^-24); and the forward, inference
    backward and training backward, fed the deterministic env, match the oracle
    evaluated on that same env at the usual bars."""
    rng = np.random.default_rng(1000 + lmax * 10 + U)
    degrees = np.floor(rng.pareto(1.2, size=160) * 6).astype(np.int64)
    degrees[rng.choice(160, 40, replace=False)] = 0
    degrees[7] = 3001 if U <= 64 else 1200
    degrees = np.minimum(degrees, 3001)
    _note(f"[gpu] skewed degrees lmax={lmax} U={U}: E={int(degrees.sum())}, max={int(degrees.max())}, "
          f"empty={int((degrees == 0).sum())}")
    row_ptr, x, w, y, pw, g = _synthetic(lmax, full, U, degrees, seed=5 + lmax + U)
    rp, xd, wd, yd, pwd, gd = (_t(a) for a in (row_ptr, x, w, y, pw, g))
    # env: deterministic mode bit-exact, fast mode within the summation bound
    det = at.allegro_env_embed(_plan(at, lmax, U, full, det=True), rp, wd, yd)
    env32 = otp.env_embed_fp32_replay(row_ptr, w, y)
    assert np.array_equal(det.cpu().numpy().view(np.uint32), env32.view(np.uint32))
    plan = _plan(at, lmax, U, full)
    fast = at.allegro_env_embed(plan, rp, wd, yd).cpu().numpy().astype(np.float64)
    abs_sum = otp.env_embed(row_ptr, np.abs(w), np.abs(y))
    n_seg = np.diff(row_ptr).astype(np.float64)[:, None, None]
    gamma = n_seg * 2.0 ** -24 / (1 - n_seg * 2.0 ** -24)
    assert np.all(np.abs(fast - otp.env_embed(row_ptr, w, y)) <= gamma * abs_sum + 1e-30)
    # the rest on the deterministic env, against the oracle on the same env values
    out = at.allegro_tp_forward(plan, rp, xd, det, pwd)
    grads = at.allegro_tp_backward(plan, rp, xd, det, pwd, gd, wd, yd)
    (gx, genv, gw, gy, gpw), _ = _train(at, plan, rp, xd, det, pwd, gd, wd, yd)
    t = otp.TensorProduct(lmax, full)
    ref_out = t.forward(row_ptr, x, env32, pw)
    ref_g = t.backward(row_ptr, x, env32, pw, g, w, y)
    errs = {"out": block_rel_err(out.cpu().numpy(), ref_out, t.x_slices)}
    for name, got, ref, blocks in (("grad_x", grads[0], ref_g[0], t.x_slices),
                                   ("grad_env", grads[1], ref_g[1], t.env_slices),
                                   ("grad_w", grads[2], ref_g[2], None), ("grad_Y", grads[3], ref_g[3], t.env_slices),
                                   ("train grad_env", genv, ref_g[1], t.env_slices),
                                   ("train grad_Y", gy, ref_g[3], t.env_slices)):
        errs[name] = block_rel_err(got.cpu().numpy(), ref, blocks)
    errs["grad_path_w"] = block_rel_err(gpw.cpu().numpy(), t.path_weight_grad(row_ptr, x, env32, g))
    _note(f"skewed lmax{lmax} U{U}: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    assert errs["out"] <= FWD_TOL
    assert all(v <= BWD_TOL for k, v in errs.items() if k != "out"), errs
    assert block_rel_err(gx.cpu().numpy(), ref_g[0], t.x_slices) <= BWD_TOL


def test_no_edges_gives_zero_env_and_grad_env(at):
    _note("[gpu] E = 0 with N = 4")
    plan = _plan(at, 2, 64, True)
    rp = torch.zeros(5, dtype=torch.int64, device=DEV)
    w = torch.empty((0, 64), device=DEV)
    y = torch.empty((0, 9), device=DEV)
    x = torch.empty((0, 64, 18), device=DEV)
    env = at.allegro_env_embed(plan, rp, w, y, env=torch.full((4, 64, 9), 7.0, device=DEV))
    pw = torch.ones((plan.n_paths, 64), device=DEV)
    outs = (torch.empty_like(x), torch.full((4, 64, 9), 7.0, device=DEV), torch.empty_like(w), torch.empty_like(y))
    gx, genv, gw, gy = at.allegro_tp_backward(plan, rp, x, env, pw, x, w, y, outs=outs)
    out = at.allegro_tp_forward(plan, rp, x, env, pw)
    torch.cuda.synchronize()
    assert out.shape == (0, 64, 18)
    assert torch.count_nonzero(env).item() == 0 and torch.count_nonzero(genv).item() == 0


def test_validate_rejects_bad_csr(at):
    _note("[gpu] CSR validation")
    plan = _plan(at, 1, 16, False, validate=True)
    w = torch.zeros((6, 16), device=DEV)
    y = torch.zeros((6, 4), device=DEV)
    for bad in ([0, 4, 2, 6], [1, 2, 4, 6], [0, 2, 4, 5]):
        rp = torch.tensor(bad, dtype=torch.int64, device=DEV)
        with pytest.raises(at.AllegroError) as ex:
            at.allegro_env_embed(plan, rp, w, y)
        assert ex.value.code == at.ALLEGRO_E_INVALID
    rp = torch.tensor([0, 2, 4, 6], dtype=torch.int64, device=DEV)
    at.allegro_env_embed(plan, rp, w, y)
    torch.cuda.synchronize()


# ------------------------------------------------- full sizes, sampled segments

def _sampled_check(at, name, n_samples=24):
    graph = workloads.make_graph(name)
    cfg = graph.config
    _note(f"[gpu] {name}: N={graph.n_atoms} E={graph.n_edges} U={cfg.U} lmax={cfg.lmax} (sampled)")
    plan = _plan(at, cfg.lmax, cfg.U, cfg.full_parity)
    x, w, g = workloads.device_features(cfg, graph.n_edges, DEV)
    pw = workloads.path_weights(cfg)
    rp, yd, pwd = _t(graph.row_ptr), _t(graph.Y), _t(pw)
    env = at.allegro_env_embed(plan, rp, w, yd)
    out = at.allegro_tp_forward(plan, rp, x, env, pwd)
    torch.cuda.synchronize()
    rng = np.random.default_rng(cfg.index)
    centers = np.unique(np.concatenate([[0, graph.n_atoms - 1], rng.integers(0, graph.n_atoms, n_samples)]))
    segs = [(int(graph.row_ptr[n]), int(graph.row_ptr[n + 1])) for n in centers]
    idx = torch.as_tensor(np.concatenate([np.arange(s, e) for s, e in segs]), device=DEV)
    local_rp = np.concatenate([[0], np.cumsum([e - s for s, e in segs])]).astype(np.int64)
    xs, ws, gs = x[idx].cpu().numpy(), w[idx].cpu().numpy(), g[idx].cpu().numpy()
    ys = graph.Y[idx.cpu().numpy()]
    env_s = env[torch.as_tensor(centers, device=DEV)].cpu().numpy()
    out_s = out[idx].cpu().numpy()
    del out
    grads = at.allegro_tp_backward(plan, rp, x, env, pwd, g, w, yd)
    torch.cuda.synchronize()
    cidx = torch.as_tensor(centers, device=DEV)
    gx_s, genv_s = grads[0][idx].cpu().numpy(), grads[1][cidx].cpu().numpy()
    gw_s, gy_s = grads[2][idx].cpu().numpy(), grads[3][idx].cpu().numpy()
    del grads, x, w, g
    torch.cuda.empty_cache()
    t, *ref = _oracle(cfg.lmax, cfg.full_parity, local_rp, xs, ws, ys, pw, gs)
    _compare(t, (env_s, out_s, (gx_s, genv_s, gw_s, gy_s)), ref, f"{name}[{len(centers)} segments]")


@pytest.mark.parametrize("name", ["headline", "high_order", "large"])
def test_full_size_sampled_segments(at, name):
    _sampled_check(at, name)


# ------------------------------------------------ spherical harmonics of edges

def _sh_vectors(n, seed):
    rng = np.random.default_rng(seed)
    v = rng.standard_normal((n, 3)) * rng.uniform(0.3, 6.0, (n, 1))
    # axis-aligned and near-polar directions, tiny and large lengths
    special = np.array([[0, 0, 1], [0, 0, -1], [1, 0, 0], [0, -1, 0], [1e-9, 0, 1], [0, 1e-12, -3],
                        [1e-3, 2e-3, 1e-3], [4e2, -3e2, 5e2]], dtype=np.float64)
    return np.concatenate([special, v])


@pytest.mark.parametrize("lmax", [1, 2, 3])
def test_sh_forward_and_backward(at, lmax):
    from oracle import sh as osh

    _note(f"[gpu] harmonics lmax={lmax}")
    plan = _plan(at, lmax, 64, True)
    vec = _sh_vectors(5000, 40 + lmax)
    d2 = (lmax + 1) ** 2
    gy = np.random.default_rng(lmax).standard_normal((len(vec), d2)).astype(np.float32)
    vd = _t(vec)
    y = at.allegro_sh_forward(plan, vd).cpu().numpy()
    gv = at.allegro_sh_backward(plan, vd, _t(gy)).cpu().numpy()
    ref_y = osh.sh_real_all(lmax, vec)
    # evaluated in fp64 and rounded once to fp32: within one fp32 rounding of the fp64 value
    assert np.all(np.abs(y - ref_y) <= 2.0 ** -23 * np.abs(ref_y) + 1e-12)
    ref_g = osh.sh_backward(lmax, vec, gy)
    err = block_rel_err(gv, ref_g)
    _note(f"harmonics lmax={lmax}: grad_vec err={err:.2e}")
    # both sides differentiate exactly in fp64 and contract the same fp32 grad_Y in fp64
    assert err <= 1e-12


def test_sh_headline_vectors_sampled(at):
    from oracle import sh as osh

    graph = workloads.make_graph("headline")
    _note(f"[gpu] harmonics of the headline edges: E={graph.n_edges}")
    plan = _plan(at, 2, 64, True)
    vd = _t(graph.vec)
    y = at.allegro_sh_forward(plan, vd)
    gy = torch.randn((graph.n_edges, 9), generator=torch.Generator(device=DEV).manual_seed(3), device=DEV)
    gv = at.allegro_sh_backward(plan, vd, gy)
    torch.cuda.synchronize()
    yh, gvh, vec = y.cpu().numpy(), gv.cpu().numpy(), graph.vec
    # every edge: sum_m Y_lm^2 = 2l + 1 and r . grad_vec = 0 (Y depends on the direction only)
    for l in range(3):
        norm = np.sum(yh[:, l * l:(l + 1) ** 2].astype(np.float64) ** 2, axis=1)
        assert np.max(np.abs(norm - (2 * l + 1))) <= 1e-6 * (2 * l + 1)
    radial = np.abs(np.sum(vec * gvh, axis=1))
    assert np.max(radial) <= 1e-12 * np.max(np.abs(gvh) * np.linalg.norm(vec, axis=1, keepdims=True))
    # sampled edges against the oracle
    idx = np.random.default_rng(9).integers(0, graph.n_edges, 4096)
    ref_y = osh.sh_real_all(2, vec[idx])
    assert np.all(np.abs(yh[idx] - ref_y) <= 2.0 ** -23 * np.abs(ref_y) + 1e-12)
    ref_g = osh.sh_backward(2, vec[idx], gy.cpu().numpy()[idx])
    assert block_rel_err(gvh[idx], ref_g) <= 1e-12


# ------------------------------------------ training backward (path weights)

def _train(at, plan, rp, x, env, pw, g, w, y):
    """The training backward into outputs filled with NaN, so that an element the
    kernels leave unwritten fails every comparison (the workspace too: rows it
    does not write stay NaN)."""
    n = rp.numel() - 1
    ws = torch.full((at.allegro_tp_backward_workspace(plan, n) // 4,), float("nan"), device=DEV).view(torch.uint8)
    outs = tuple(torch.full_like(a, float("nan")) for a in (x, env, w, y, pw))
    res = at.allegro_tp_backward_train(plan, rp, x, env, pw, g, w, y, outs=outs, workspace=ws)
    torch.cuda.synchronize()
    return res, ws


def _same_bits(a, b):
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


@pytest.mark.parametrize("case", ["tiny", "small"] + [f"edge{i}" for i in range(len(EDGE_CASES))])
def test_train_backward_parity(at, case):
    if case.startswith("edge"):
        lmax, full, U, degrees = EDGE_CASES[int(case[4:])]
        data = _synthetic(lmax, full, U, degrees, seed=7 + lmax * 10 + U)
    else:
        graph = workloads.make_graph(case)
        cfg = graph.config
        lmax, full, U = cfg.lmax, cfg.full_parity, cfg.U
        x, w, pw, g = workloads.host_features(cfg, graph.n_edges)
        data = (graph.row_ptr, x, w, graph.Y, pw, g)
    _note(f"[gpu] training backward {case}: lmax={lmax} full={full} U={U}")
    plan = _plan(at, lmax, U, full)
    rp, xd, wd, yd, pwd, gd = (_t(a) for a in data)
    env = at.allegro_env_embed(plan, rp, wd, yd)
    base = at.allegro_tp_backward(plan, rp, xd, env, pwd, gd, wd, yd)
    (gx, genv, gw, gy, gpw), _ = _train(at, plan, rp, xd, env, pwd, gd, wd, yd)
    # the training backward splits the work differently from the inference
    # backward (other wave counts; at lmax 3 a per-center matrix for grad_x and
    # per-center products for the segment sums), so its gradients agree with the
    # inference ones to fp32 rounding; both match the oracle
    t = otp.TensorProduct(lmax, full)
    renv = otp.env_embed(data[0], data[2], data[3])
    ref = t.backward(data[0], data[1], renv, data[4], data[5], data[2], data[3])
    for got, r, blocks in zip((gx, genv, gw, gy), ref, (t.x_slices, t.env_slices, None, t.env_slices)):
        assert block_rel_err(got.cpu().numpy(), r, blocks) <= BWD_TOL
    for got, b in zip((gx, genv, gw, gy), base):
        assert block_rel_err(got.cpu().numpy(), b.cpu().numpy()) <= BWD_TOL
    ref = t.path_weight_grad(data[0], data[1], otp.env_embed(data[0], data[2], data[3]), data[5])
    err = block_rel_err(gpw.cpu().numpy(), ref)
    _note(f"training backward {case}: grad_path_w err={err:.2e}")
    assert err <= BWD_TOL
    # deterministic: a second call gives the same bits
    (_, _, _, _, gpw2), _ = _train(at, plan, rp, xd, env, pwd, gd, wd, yd)
    assert _same_bits(gpw, gpw2)


def test_train_backward_without_edges(at):
    _note("[gpu] training backward with E = 0 (N = 3) and N = 0")
    plan = _plan(at, 2, 32, False)
    pw = torch.ones((plan.n_paths, 32), device=DEV)
    x = torch.empty((0, 32, plan.d1), device=DEV)
    w, y = torch.empty((0, 32), device=DEV), torch.empty((0, plan.d2), device=DEV)
    for n in (3, 0):
        rp = torch.zeros(n + 1, dtype=torch.int64, device=DEV)
        env = torch.randn((n, 32, plan.d2), device=DEV)
        outs = (torch.empty_like(x), torch.full_like(env, 5.0), torch.empty_like(w), torch.empty_like(y),
                torch.full_like(pw, 9.0))
        (_, genv, _, _, gpw), _ = (at.allegro_tp_backward_train(plan, rp, x, env, pw, x, w, y, outs=outs), None)
        torch.cuda.synchronize()
        assert torch.count_nonzero(gpw).item() == 0 and torch.count_nonzero(genv).item() == 0


def test_handover_timeout_is_reported_and_ends(at, monkeypatch):
    """With the handover waits of the lmax-3 matrix-core backward forced to give
    up at once (a plan created under ALLEGRO_SIMULATE_HANDOVER_TIMEOUT), the
    kernel still runs to its end: a validating plan reports ALLEGRO_E_TIMEOUT
    (both entry points), a plain one returns; a normal plan afterwards is exact."""
    lmax, full, U, degrees = 3, True, 64, [1, 0, 9, 70, 33]
    data = _synthetic(lmax, full, U, degrees, seed=41)
    rp, xd, wd, yd, pwd, gd = (_t(a) for a in data)
    _note("[gpu] handover timeout forced from the host: lmax 3, U 64")
    monkeypatch.setenv("ALLEGRO_SIMULATE_HANDOVER_TIMEOUT", "1")
    stalled = _plan(at, lmax, U, full, validate=True)
    stalled_plain = _plan(at, lmax, U, full)
    monkeypatch.delenv("ALLEGRO_SIMULATE_HANDOVER_TIMEOUT")
    normal = _plan(at, lmax, U, full, validate=True)
    env = at.allegro_env_embed(normal, rp, wd, yd)
    with pytest.raises(at.AllegroError) as ex:
        _train(at, stalled, rp, xd, env, pwd, gd, wd, yd)
    assert ex.value.code == at.ALLEGRO_E_TIMEOUT and "ran out" in str(ex.value)
    with pytest.raises(at.AllegroError) as ex:
        at.allegro_tp_backward_train_noalloc(stalled, rp, xd, env, pwd, gd, wd, yd)
    assert ex.value.code == at.ALLEGRO_E_TIMEOUT
    _train(at, stalled_plain, rp, xd, env, pwd, gd, wd, yd)  # returns; its outputs are not valid
    (gx, genv, gw, gy, gpw), _ = _train(at, normal, rp, xd, env, pwd, gd, wd, yd)
    t = otp.TensorProduct(lmax, full)
    renv = otp.env_embed(data[0], data[2], data[3])
    ref = t.backward(data[0], data[1], renv, data[4], data[5], data[2], data[3])
    for got, r, blocks in zip((gx, genv, gw, gy), ref, (t.x_slices, t.env_slices, None, t.env_slices)):
        assert block_rel_err(got.cpu().numpy(), r, blocks) <= BWD_TOL
    assert block_rel_err(gpw.cpu().numpy(), t.path_weight_grad(data[0], data[1], renv, data[5])) <= BWD_TOL


@pytest.mark.parametrize("lmax,U,full", [(1, 16, False), (3, 16, True), (3, 128, True)])
def test_train_backward_rejects_small_workspace(at, lmax, U, full):
    """Per-center rows (lmax < 3) or the matrix-core kernel's per-wave rows (lmax 3):
    a workspace one float4 short of the size the query gives is rejected before any launch."""
    plan = _plan(at, lmax, U, full)
    rp = torch.tensor([0, 2], dtype=torch.int64, device=DEV)
    x = torch.zeros((2, U, plan.d1), device=DEV)
    w, y = torch.zeros((2, U), device=DEV), torch.zeros((2, plan.d2), device=DEV)
    env, pw = torch.zeros((1, U, plan.d2), device=DEV), torch.zeros((plan.n_paths, U), device=DEV)
    ws = torch.empty(at.allegro_tp_backward_workspace(plan, 1) - 16, dtype=torch.uint8, device=DEV)
    with pytest.raises(at.AllegroError) as ex:
        at.allegro_tp_backward_train(plan, rp, x, env, pw, x, w, y, workspace=ws)
    assert ex.value.code == at.ALLEGRO_E_INVALID and "workspace" in str(ex.value)


@pytest.mark.parametrize("name", ["headline", "high_order", "large"])
def test_train_backward_full_size(at, name, n_samples=16):
    """Full size, sampled: grad_x and each sampled center's path-weight rows
    against the oracle, and grad_path_w against the fp64 sum of the partial rows
    the workspace holds.  At lmax < 3 those are per-center rows ([N][P][U]); at
    lmax 3 the matrix-core kernel writes one [U][P] row per round of its waves
    (each the sum over the centers that round visited), so a center's own row is
    taken from a second call on a one-center CSR that points into the same
    tensors (its grad_path_w is that row)."""
    graph = workloads.make_graph(name)
    cfg = graph.config
    _note(f"[gpu] training backward {name}: N={graph.n_atoms} E={graph.n_edges} (sampled)")
    plan = _plan(at, cfg.lmax, cfg.U, cfg.full_parity)
    x, w, g = workloads.device_features(cfg, graph.n_edges, DEV)
    pw = workloads.path_weights(cfg)
    rp, yd, pwd = _t(graph.row_ptr), _t(graph.Y), _t(pw)
    env = at.allegro_env_embed(plan, rp, w, yd)
    (gx, genv, gw, gy, gpw), ws = _train(at, plan, rp, x, env, pwd, g, w, yd)
    # every element written (the outputs start as NaN)
    for name_, a in (("grad_x", gx), ("grad_env", genv), ("grad_w", gw), ("grad_Y", gy), ("grad_path_w", gpw)):
        assert not bool(torch.isnan(a).any()), f"{name_} has unwritten elements"
    n, cols = graph.n_atoms, plan.n_paths * cfg.U
    wsf = ws.view(torch.float32)
    if cfg.lmax >= 3:
        # rows written: a prefix of whole [U][P] rows, the rest still NaN
        rows = wsf.view(-1, cfg.U, plan.n_paths)
        written = ~torch.isnan(rows).view(rows.shape[0], -1).any(dim=1)
        n_rows = int(written.sum())
        assert n_rows >= 1 and bool(written[:n_rows].all()) and not bool(written[n_rows:].any())
        part = rows[:n_rows].permute(0, 2, 1)
    else:
        n_rows = n
        part = wsf[: n * cols].view(n, plan.n_paths, cfg.U)
    ph = np.ascontiguousarray(part.cpu().numpy()).astype(np.float64).reshape(n_rows, cols)
    del part, ws, wsf
    ws1 = torch.empty(at.allegro_tp_backward_workspace(plan, 1), dtype=torch.uint8, device=DEV)
    rng = np.random.default_rng(cfg.index + 50)
    centers = np.unique(np.concatenate([[0, n - 1], rng.integers(0, n, n_samples)]))
    t = otp.TensorProduct(cfg.lmax, cfg.full_parity)
    for c in centers:
        s, e = int(graph.row_ptr[c]), int(graph.row_ptr[c + 1])
        xs, ws_, gs = x[s:e].cpu().numpy(), w[s:e].cpu().numpy(), g[s:e].cpu().numpy()
        local = np.array([0, e - s], np.int64)
        env_c = otp.env_embed(local, ws_, graph.Y[s:e])
        ref = t.path_weight_grad(local, xs, env_c, gs)
        if cfg.lmax >= 3:
            before = [a[s:e].clone() for a in (gx, gw, gy)]
            o_env = torch.full_like(genv[c:c + 1], float("nan"))
            o_pw = torch.full_like(gpw, float("nan"))
            at.allegro_tp_backward_train(plan, rp[c:c + 2], x, env[c:c + 1], pwd, g, w, yd,
                                         outs=(gx, o_env, gw, gy, o_pw), workspace=ws1)
            torch.cuda.synchronize()
            for a, b in zip((gx, gw, gy), before):
                assert _same_bits(a[s:e], b), c  # the same rows as in the full call
            assert _same_bits(o_env[0], genv[c]), c
            row = o_pw.cpu().numpy()
        else:
            row = ph[c].reshape(plan.n_paths, cfg.U)
        assert block_rel_err(row, ref) <= BWD_TOL, c
        ref_gx = t.backward(local, xs, env_c, pw, gs, ws_, graph.Y[s:e])[0]
        assert block_rel_err(gx[s:e].cpu().numpy(), ref_gx, t.x_slices) <= BWD_TOL, c
    del gx, genv, gw, gy
    total = ph.sum(axis=0)
    if cfg.lmax >= 3:
        depth = n_rows + 1  # one fixed-order sum over the rows
    else:
        # recursive-summation bound: at most ceil(ceil(N / 128) / 4) + 130 sequential fp32 additions
        depth = -(-(-(-n // 128)) // 4) + 130
    bound = 1.01 * depth * 2.0 ** -24 * np.abs(ph).sum(axis=0)
    got = gpw.cpu().numpy().reshape(cols).astype(np.float64)
    assert np.all(np.abs(got - total) <= bound)


def test_scalar_path_weights_broadcast(at):
    """One scalar weight per path, passed broadcast over the channels; its gradient is grad_path_w summed over u."""
    graph = workloads.make_graph("small")
    cfg = graph.config
    x, w, _, g = workloads.host_features(cfg, graph.n_edges)
    _note("[gpu] scalar path weights broadcast over channels, small")
    scal = np.random.default_rng(31).standard_normal((workloads.dims(cfg.lmax, cfg.full_parity)[2], 1))
    pw = np.ascontiguousarray(np.broadcast_to(scal, (scal.shape[0], cfg.U))).astype(np.float32)
    plan = _plan(at, cfg.lmax, cfg.U, cfg.full_parity)
    rp, xd, wd, yd, pwd, gd = (_t(a) for a in (graph.row_ptr, x, w, graph.Y, pw, g))
    env = at.allegro_env_embed(plan, rp, wd, yd)
    out = at.allegro_tp_forward(plan, rp, xd, env, pwd)
    (_, _, _, _, gpw), _ = _train(at, plan, rp, xd, env, pwd, gd, wd, yd)
    t = otp.TensorProduct(cfg.lmax, cfg.full_parity)
    renv = otp.env_embed(graph.row_ptr, w, graph.Y)
    assert block_rel_err(out.cpu().numpy(), t.forward(graph.row_ptr, x, renv, pw), t.x_slices) <= FWD_TOL
    ref_scalar = t.path_weight_grad(graph.row_ptr, x, renv, g).sum(axis=1)
    got_scalar = gpw.cpu().numpy().astype(np.float64).sum(axis=1)
    assert block_rel_err(got_scalar, ref_scalar) <= BWD_TOL


@pytest.mark.parametrize("name", ["headline", "high_order", "large"])
def test_deterministic_env_full_size_sampled(at, name, n_samples=32):
    """Deterministic env at full size: sampled centers bit-equal to the fp32 sequential replay."""
    graph = workloads.make_graph(name)
    cfg = graph.config
    _note(f"[gpu] deterministic env {name} (sampled)")
    plan = _plan(at, cfg.lmax, cfg.U, cfg.full_parity, det=True)
    _, w, _ = workloads.device_features(cfg, graph.n_edges, DEV)
    env = at.allegro_env_embed(plan, _t(graph.row_ptr), w, _t(graph.Y))
    torch.cuda.synchronize()
    rng = np.random.default_rng(cfg.index + 70)
    centers = np.unique(np.concatenate([[0, graph.n_atoms - 1], rng.integers(0, graph.n_atoms, n_samples)]))
    for c in centers:
        s, e = int(graph.row_ptr[c]), int(graph.row_ptr[c + 1])
        ref = otp.env_embed_fp32_replay(np.array([0, e - s], np.int64), w[s:e].cpu().numpy(), graph.Y[s:e])
        assert np.array_equal(env[c:c + 1].cpu().numpy().view(np.uint32), ref.view(np.uint32)), c


def test_step_replays_in_a_hip_graph(at):
    """The whole step (harmonics, embedding, forward, training backward, harmonics VJP)
    captured once into a HIP graph and replayed several times, with eager work and
    synchronisation in between; every replay must equal the eager result bit for bit."""
    graph = workloads.make_graph("small")
    cfg = graph.config
    x, w, pw, g = workloads.host_features(cfg, graph.n_edges)
    _note("[gpu] HIP graph replay of the step, small")
    plan = _plan(at, cfg.lmax, cfg.U, cfg.full_parity)
    rp, xd, wd, pwd, gd, vec = (_t(a) for a in (graph.row_ptr, x, w, pw, g, graph.vec))
    n, e = graph.n_atoms, graph.n_edges
    y = torch.empty((e, plan.d2), device=DEV)
    env = torch.empty((n, cfg.U, plan.d2), device=DEV)
    out = torch.empty_like(xd)
    outs = (torch.empty_like(xd), torch.empty_like(env), torch.empty_like(wd), torch.empty_like(y),
            torch.empty_like(pwd))
    gvec = torch.empty((e, 3), device=DEV, dtype=torch.float64)
    ws = torch.empty(at.allegro_tp_backward_workspace(plan, n), dtype=torch.uint8, device=DEV)

    def step():
        at.allegro_sh_forward(plan, vec, Y=y)
        at.allegro_env_embed(plan, rp, wd, y, env=env)
        at.allegro_tp_forward(plan, rp, xd, env, pwd, out=out)
        at.allegro_tp_backward_train(plan, rp, xd, env, pwd, gd, wd, y, outs=outs, workspace=ws)
        at.allegro_sh_backward(plan, vec, outs[3], grad_vec=gvec)

    results = (y, env, out, *outs, gvec)
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
        torch.cuda.synchronize()
        hip_graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(results, eager):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), rep
