"""Pins of the oracle's spherical harmonics and Wigner matrices.

* complex harmonics against scipy.special (an independent library routine);
* real harmonics against the Cartesian closed forms written out below;
* addition theorem with numpy's Legendre polynomials; quadrature
  orthonormality; parity Y(-r) = (-1)^l Y(r);
* Wigner matrices: orthogonality, the homomorphism D(R1 R2) = D(R1) D(R2), and
  D^1 = P R P^T for the permutation (x, y, z) -> (y, z, x).
"""

from math import pi, sqrt

import numpy as np
import pytest

from oracle import sh, wigner


def _dirs(n, seed=3):
    v = np.random.default_rng(seed).standard_normal((n, 3))
    return v / np.linalg.norm(v, axis=1, keepdims=True)


def test_complex_against_scipy():
    special = pytest.importorskip("scipy.special")
    if not hasattr(special, "sph_harm_y"):
        pytest.skip("scipy without sph_harm_y")
    v = _dirs(50)
    theta = np.arccos(np.clip(v[:, 2], -1, 1))
    phi = np.arctan2(v[:, 1], v[:, 0])
    for l in range(5):
        ours = sh.sh_complex(l, v)
        for m in range(-l, l + 1):
            ref = special.sph_harm_y(l, m, theta, phi)
            np.testing.assert_allclose(ours[:, m + l], ref, atol=1e-12)


def test_real_cartesian_closed_forms():
    v = _dirs(64)
    x, y, z = v[:, 0], v[:, 1], v[:, 2]
    expect = {
        0: [np.ones_like(x)],
        1: [sqrt(3) * y, sqrt(3) * z, sqrt(3) * x],
        2: [sqrt(15) * x * y, sqrt(15) * y * z, sqrt(5) / 2 * (3 * z ** 2 - 1), sqrt(15) * x * z,
            sqrt(15) / 2 * (x ** 2 - y ** 2)],
    }
    for l, cols in expect.items():
        np.testing.assert_allclose(sh.sh_real(l, v), np.stack(cols, axis=1), atol=1e-13)


def test_addition_theorem_and_parity():
    a, b = _dirs(40, 1), _dirs(40, 2)
    cosg = np.sum(a * b, axis=1)
    for l in range(6):
        ya, yb = sh.sh_real(l, a), sh.sh_real(l, b)
        pl = np.polynomial.legendre.legval(cosg, [0] * l + [1])
        np.testing.assert_allclose(np.sum(ya * yb, axis=1), (2 * l + 1) * pl, atol=1e-12)
        np.testing.assert_allclose(sh.sh_real(l, -a), (-1) ** l * ya, atol=1e-13)


def test_quadrature_orthonormality():
    nodes, weights = np.polynomial.legendre.leggauss(16)
    n_phi = 32
    phi = (np.arange(n_phi) + 0.5) * 2 * pi / n_phi
    ct, ph = np.meshgrid(nodes, phi, indexing="ij")
    st = np.sqrt(1 - ct * ct)
    pts = np.stack([st * np.cos(ph), st * np.sin(ph), ct], axis=-1).reshape(-1, 3)
    wts = (weights[:, None] * np.full(n_phi, 2 * pi / n_phi)[None, :]).reshape(-1)
    y = sh.sh_real_all(4, pts)
    gram = (y * wts[:, None]).T @ y / (4 * pi)
    np.testing.assert_allclose(gram, np.eye(y.shape[1]), atol=1e-12)


def test_wigner_properties():
    rng = np.random.default_rng(11)
    r1, r2 = wigner.random_rotation(rng), wigner.random_rotation(rng)
    for l in range(5):
        d1, d2, d12 = (wigner.wigner_d_real(l, r) for r in (r1, r2, r1 @ r2))
        np.testing.assert_allclose(d1 @ d1.T, np.eye(2 * l + 1), atol=1e-11)
        np.testing.assert_allclose(d12, d1 @ d2, atol=1e-11)
    perm = np.eye(3)[[1, 2, 0]]  # (x, y, z) -> (y, z, x)
    np.testing.assert_allclose(wigner.wigner_d_real(1, r1), perm @ r1 @ perm.T, atol=1e-12)


def _fd_grad(lmax, v, h=1e-4):
    """Fourth-order central differences of the values, step scaled by |r| (a pin of the
    exact gradient: truncation O(h^4) and rounding O(eps/h) stay near 1e-11 relative)."""
    scale = np.linalg.norm(v, axis=-1, keepdims=True)
    out = np.zeros(v.shape[:-1] + ((lmax + 1) ** 2, 3))
    for k in range(3):
        step = np.zeros_like(v)
        step[..., k] = h * scale[..., 0]
        f = [sh.sh_real_all(lmax, v + c * step) for c in (2, 1, -1, -2)]
        out[..., k] = (-f[0] + 8 * f[1] - 8 * f[2] + f[3]) / (12 * h * scale)
    return out


def _vectors(n, seed):
    rng = np.random.default_rng(seed)
    v = rng.standard_normal((n, 3)) * rng.uniform(0.3, 6.0, (n, 1))
    special = np.array([[0, 0, 1.5], [0, 0, -2.0], [1, 0, 0], [0, -1, 0], [1e-7, 0, 1], [1e-3, 2e-3, 1e-3]])
    return np.concatenate([special, v])


def test_gradient_matches_finite_differences():
    v = _vectors(60, 8)
    for lmax in (1, 2, 3, 4):
        exact = sh.sh_real_all_grad(lmax, v)
        fd = _fd_grad(lmax, v)
        scale = np.abs(exact).max(axis=(1, 2), keepdims=True)
        assert np.max(np.abs(exact - fd) / scale) < 1e-9, lmax


def test_gradient_closed_forms_l1_l2():
    rng = np.random.default_rng(4)
    v = rng.standard_normal((30, 3)) * rng.uniform(0.5, 5.0, (30, 1))
    grad = sh.sh_real_all_grad(2, v)
    r = np.linalg.norm(v, axis=1)
    u = v / r[:, None]
    eye = np.eye(3)
    # du_a/dr = (e_a - u_a u) / |r|
    du = [(eye[a][None, :] - u[:, a:a + 1] * u) / r[:, None] for a in range(3)]
    # l = 1: Y = sqrt3 (u_y, u_z, u_x)
    for col, axis in ((1, 1), (2, 2), (3, 0)):
        np.testing.assert_allclose(grad[:, col, :], sqrt(3) * du[axis], atol=1e-13)
    # l = 2: sqrt15 u_x u_y, sqrt15 u_y u_z, sqrt5/2 (3 u_z^2 - 1), sqrt15 u_x u_z, sqrt15/2 (u_x^2 - u_y^2)
    x, y, z = (u[:, a:a + 1] for a in range(3))
    expect = [sqrt(15) * (y * du[0] + x * du[1]), sqrt(15) * (z * du[1] + y * du[2]), sqrt(5) / 2 * 6 * z * du[2],
              sqrt(15) * (z * du[0] + x * du[2]), sqrt(15) / 2 * (2 * x * du[0] - 2 * y * du[1])]
    for c, e in enumerate(expect):
        np.testing.assert_allclose(grad[:, 4 + c, :], e, atol=1e-13)
    # Y is homogeneous of degree 0, so r . grad Y = 0 for every component; Y_0 is constant
    grad3 = sh.sh_real_all_grad(4, v)
    np.testing.assert_allclose(np.einsum("ek,ejk->ej", v, grad3), 0.0, atol=1e-13)
    np.testing.assert_allclose(grad3[:, 0, :], 0.0, atol=0.0)


def test_gradient_equivariance():
    rng = np.random.default_rng(5)
    rot = wigner.random_rotation(rng)
    v = rng.standard_normal((20, 3))
    lmax = 3
    # Y(R r) = D Y(r)  =>  J(R r) R = D J(r)   (J = dY/dr)
    blocks = [(l, 1 if l % 2 == 0 else -1) for l in range(lmax + 1)]
    d = wigner.wigner_d_blocks(blocks, rot)
    j_rot = sh.sh_real_all_grad(lmax, v @ rot.T)
    j = sh.sh_real_all_grad(lmax, v)
    np.testing.assert_allclose(np.einsum("ejk,kl->ejl", j_rot, rot), np.einsum("ij,ejk->eik", d, j), atol=1e-10)


def test_backward_directional_differences():
    """sh_backward against the loss L(r) = <grad_Y, Y(r)> alone: for a random direction d
    per edge, <grad_vec, d> equals dL(r + t d)/dt at t = 0 (fourth-order differences
    of the values; no Jacobian involved)."""
    rng = np.random.default_rng(6)
    v = _vectors(200, 9)
    for lmax in (1, 2, 3):
        gy = rng.standard_normal((len(v), (lmax + 1) ** 2))
        d = rng.standard_normal(v.shape)
        h = 1e-4 * np.linalg.norm(v, axis=1, keepdims=True)
        loss = [np.sum(gy * sh.sh_real_all(lmax, v + c * h * d), axis=1) for c in (2, 1, -1, -2)]
        fd = (-loss[0] + 8 * loss[1] - 8 * loss[2] + loss[3]) / (12 * h[:, 0])
        got = np.sum(sh.sh_backward(lmax, v, gy) * d, axis=1)
        scale = np.linalg.norm(gy, axis=1) * np.linalg.norm(d, axis=1) / np.linalg.norm(v, axis=1)
        assert np.max(np.abs(got - fd) / scale) < 1e-9, lmax
