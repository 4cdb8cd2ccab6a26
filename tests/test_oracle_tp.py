"""Pins of the oracle's embedding and tensor product (forward and VJP).

* nested loops against the per-path einsum form (two independent codings);
* equivariance: rotating every edge vector (so Y -> D Y, env -> D env) and
  every x block by its Wigner matrix rotates every output block by D^{l3};
  under inversion every block picks up its parity, which pins the path
  selection rule;
* special paths: 0e x 0e -> 0e is a product, 1o x 1o -> 0e the dot product
  over sqrt 3, 1o x 1o -> 1e the cross product over sqrt 2;
* the VJP: exact adjoint identities of a bilinear map and central finite
  differences through x, env, w and Y;
* the embedding: brute-force loops, empty segments, and the fp32 replay;
* the path-weight gradient: out is linear in W, so each grad_W[p, u] equals
  <g, out> with W the one-hot e_pu (the forward, pinned above).
"""

from math import sqrt

import numpy as np
import pytest

import workloads
from oracle import irreps, sh, tp, wigner


def _problem(lmax, full, n_ch, seed=0, n_atoms=10, box=6.0, cutoff=2.9, rot=None):
    rng = np.random.default_rng(seed)
    pos = rng.uniform(0, box, size=(n_atoms, 3))
    row_ptr, _, vec = workloads.neighbor_list(pos, box, cutoff)
    if rot is not None:
        vec = vec @ rot.T
    d1, d2, n_paths = workloads.dims(lmax, full)
    n_edges = int(row_ptr[-1])
    x = rng.standard_normal((n_edges, n_ch, d1))
    w = rng.standard_normal((n_edges, n_ch))
    W = rng.standard_normal((n_paths, n_ch))
    g = rng.standard_normal((n_edges, n_ch, d1))
    y = sh.sh_real_all(lmax, vec)
    return row_ptr, vec, x, w, W, g, y


CASES = [(1, False, 3), (2, True, 2), (3, True, 2)]


@pytest.mark.parametrize("lmax,full,n_ch", CASES)
def test_forward_loops_match_einsum(lmax, full, n_ch):
    row_ptr, _, x, w, W, _, y = _problem(lmax, full, n_ch)
    t = tp.TensorProduct(lmax, full)
    env = tp.env_embed(row_ptr, w, y)
    a = t.forward(row_ptr, x, env, W)
    b = t.forward_loops(row_ptr, x, env, W)
    assert np.abs(a - b).max() <= 1e-12 * np.abs(b).max()


@pytest.mark.parametrize("lmax,full,n_ch", CASES)
def test_backward_loops_match_einsum(lmax, full, n_ch):
    row_ptr, _, x, w, W, g, y = _problem(lmax, full, n_ch, seed=1)
    t = tp.TensorProduct(lmax, full)
    env = tp.env_embed(row_ptr, w, y)
    for a, b in zip(t.backward(row_ptr, x, env, W, g, w, y), t.backward_loops(row_ptr, x, env, W, g, w, y)):
        assert np.abs(a - b).max() <= 1e-12 * np.abs(b).max()


def test_env_embed_forms_and_empty_segments():
    rng = np.random.default_rng(5)
    degrees = np.array([3, 0, 5, 0, 1, 7])
    row_ptr = np.concatenate([[0], np.cumsum(degrees)])
    w = rng.standard_normal((row_ptr[-1], 4)).astype(np.float32)
    y = rng.standard_normal((row_ptr[-1], 9)).astype(np.float32)
    env = tp.env_embed(row_ptr, w, y)
    np.testing.assert_allclose(env, tp.env_embed_loops(row_ptr, w, y), rtol=0, atol=1e-13)
    assert np.all(env[1] == 0) and np.all(env[3] == 0)
    rep = tp.env_embed_fp32_replay(row_ptr, w, y)
    assert rep.dtype == np.float32
    np.testing.assert_allclose(rep, env, rtol=0, atol=1e-5)
    # the replay is a strict left-to-right fp32 sum: check one entry by hand
    acc = np.float32(0)
    for e in range(row_ptr[2], row_ptr[3]):
        acc = np.float32(acc + np.float32(w[e, 2] * y[e, 4]))
    assert rep[2, 2, 4] == acc


@pytest.mark.parametrize("lmax,full,n_ch", CASES)
@pytest.mark.parametrize("improper", [False, True])
def test_equivariance(lmax, full, n_ch, improper):
    rng = np.random.default_rng(21)
    rot = wigner.random_rotation(rng)
    if improper:
        rot = -rot
    t = tp.TensorProduct(lmax, full)
    row_ptr, _, x, w, W, _, y = _problem(lmax, full, n_ch, seed=2)
    _, _, _, _, _, _, y_rot = _problem(lmax, full, n_ch, seed=2, rot=rot)
    dx = wigner.wigner_d_blocks(t.x_irreps, rot)
    dy = wigner.wigner_d_blocks(t.env_irreps, rot)
    np.testing.assert_allclose(y_rot, y @ dy.T, atol=1e-10)
    out = t.forward(row_ptr, x, tp.env_embed(row_ptr, w, y), W)
    out_rot = t.forward(row_ptr, x @ dx.T, tp.env_embed(row_ptr, w, y_rot), W)
    np.testing.assert_allclose(out_rot, out @ dx.T, atol=1e-9 * np.abs(out).max())


def _only_path(t, n_ch, want):
    W = np.zeros((t.n_paths, n_ch))
    names = [tuple(irreps.irrep_name(ir) for ir in (t.x_irreps[a], t.env_irreps[b], t.x_irreps[c]))
             for a, b, c in t.paths]
    p = names.index(want)
    W[p] = np.linspace(0.5, 1.5, n_ch)
    return W, p, t.paths[p]


def test_special_paths():
    t = tp.TensorProduct(1, True)
    row_ptr, _, x, w, _, _, y = _problem(1, True, 3, seed=4)
    env = tp.env_embed(row_ptr, w, y)
    c = tp.centers_of_edges(row_ptr)
    ec = env[c]
    # 0e x 0e -> 0e
    W, p, (a, b, cc) = _only_path(t, 3, ("0e", "0e", "0e"))
    out = t.forward(row_ptr, x, env, W)
    np.testing.assert_allclose(out[:, :, 0], W[p][None] * x[:, :, 0] * ec[:, :, 0], rtol=1e-13)
    assert np.all(out[:, :, 1:] == 0)
    # 1o x 1o -> 0e: dot product / sqrt 3
    W, p, (a, b, cc) = _only_path(t, 3, ("1o", "1o", "0e"))
    out = t.forward(row_ptr, x, env, W)
    sa, sb, sc = t.x_slices[a], t.env_slices[b], t.x_slices[cc]
    dot = np.sum(x[:, :, sa] * ec[:, :, sb], axis=2)
    np.testing.assert_allclose(out[:, :, sc][:, :, 0], W[p][None] * dot / sqrt(3), rtol=1e-12, atol=1e-14)
    # 1o x 1o -> 1e: cross product / sqrt 2 in the (y, z, x) component order
    W, p, (a, b, cc) = _only_path(t, 3, ("1o", "1o", "1e"))
    out = t.forward(row_ptr, x, env, W)
    sa, sb, sc = t.x_slices[a], t.env_slices[b], t.x_slices[cc]
    to_xyz = [2, 0, 1]  # (y, z, x) -> (x, y, z)
    to_yzx = [1, 2, 0]
    cross = np.cross(x[:, :, sa][:, :, to_xyz], ec[:, :, sb][:, :, to_xyz])[:, :, to_yzx]
    np.testing.assert_allclose(out[:, :, sc], W[p][None, :, None] * cross / sqrt(2), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("lmax,full,n_ch", CASES)
def test_backward_adjoint_identities(lmax, full, n_ch):
    rng = np.random.default_rng(8)
    row_ptr, _, x, w, W, g, y = _problem(lmax, full, n_ch, seed=3)
    t = tp.TensorProduct(lmax, full)
    env = tp.env_embed(row_ptr, w, y)
    gx, genv, gw, gy = t.backward(row_ptr, x, env, W, g, w, y)
    v = rng.standard_normal(x.shape)
    eps = rng.standard_normal(env.shape)
    lhs_x = np.sum(g * t.forward(row_ptr, v, env, W))
    lhs_e = np.sum(g * t.forward(row_ptr, x, eps, W))
    assert abs(lhs_x - np.sum(gx * v)) <= 1e-11 * (abs(lhs_x) + 1)
    assert abs(lhs_e - np.sum(genv * eps)) <= 1e-11 * (abs(lhs_e) + 1)
    # embedding: <grad_env, env(dw, Y)> = <grad_w, dw> and <grad_env, env(w, dY)> = <grad_Y, dY>
    dw = rng.standard_normal(w.shape)
    dy = rng.standard_normal(y.shape)
    a = np.sum(genv * tp.env_embed(row_ptr, dw, y))
    b = np.sum(genv * tp.env_embed(row_ptr, w, dy))
    assert abs(a - np.sum(gw * dw)) <= 1e-11 * (abs(a) + 1)
    assert abs(b - np.sum(gy * dy)) <= 1e-11 * (abs(b) + 1)


def test_backward_finite_differences():
    lmax, full, n_ch = 2, True, 2
    rng = np.random.default_rng(9)
    row_ptr, _, x, w, W, g, y = _problem(lmax, full, n_ch, seed=6)
    t = tp.TensorProduct(lmax, full)

    def loss(x_, w_, y_):
        return np.sum(g * t.forward(row_ptr, x_, tp.env_embed(row_ptr, w_, y_), W))

    gx, genv, gw, gy = t.backward(row_ptr, x, tp.env_embed(row_ptr, w, y), W, g, w, y)
    h = 1e-6
    for _ in range(3):
        vx, vw, vy = rng.standard_normal(x.shape), rng.standard_normal(w.shape), rng.standard_normal(y.shape)
        fd_x = (loss(x + h * vx, w, y) - loss(x - h * vx, w, y)) / (2 * h)
        fd_w = (loss(x, w + h * vw, y) - loss(x, w - h * vw, y)) / (2 * h)
        fd_y = (loss(x, w, y + h * vy) - loss(x, w, y - h * vy)) / (2 * h)
        for fd, an in ((fd_x, np.sum(gx * vx)), (fd_w, np.sum(gw * vw)), (fd_y, np.sum(gy * vy))):
            assert abs(fd - an) <= 1e-8 * max(1.0, abs(an)), (fd, an)


@pytest.mark.parametrize("lmax,full,n_ch", CASES)
def test_path_weight_grad(lmax, full, n_ch):
    """grad_W against the forward: out is linear in W, so grad_W[p, u] = <g, out(W = e_pu)>."""
    row_ptr, _, x, w, W, g, y = _problem(lmax, full, n_ch, seed=12)
    t = tp.TensorProduct(lmax, full)
    env = tp.env_embed(row_ptr, w, y)
    gW = t.path_weight_grad(row_ptr, x, env, g)
    assert gW.shape == (t.n_paths, n_ch)
    onehot = np.zeros_like(W)
    for p in range(t.n_paths):
        for u in range(n_ch):
            onehot[p, u] = 1.0
            ref = np.sum(g * t.forward(row_ptr, x, env, onehot))
            onehot[p, u] = 0.0
            assert abs(gW[p, u] - ref) <= 1e-11 * (abs(ref) + 1), (p, u)
    # the loop form agrees; a segment-free edge set gives zero
    small = row_ptr[:4] if lmax == 3 else row_ptr
    ne = int(small[-1])
    loops = t.path_weight_grad_loops(small, x[:ne], env, g[:ne])
    assert np.abs(loops - t.path_weight_grad(small, x[:ne], env, g[:ne])).max() <= 1e-12 * (np.abs(loops).max() + 1)
    assert not t.path_weight_grad(np.zeros(3, np.int64), x[:0], env[:2], g[:0]).any()
