"""Pins of the oracle's coupling coefficients against mathematics, not against itself.

* complex CG: orthogonality in both directions, the closed forms for L = 0,
  L = l1 + l2 (stretched) and l2 = 0, the printed Condon-Shortley table
  (tests/golden/cg_condon_shortley.txt) and sympy's independent routine;
* real coupling tensors: equivariance C(D1 a, D2 b) = D3 C(a, b) with Wigner
  matrices fitted from the harmonics, proportionality to the quadrature of a
  triple product of harmonics (Gaunt integral) whenever l1 + l2 + l3 is even,
  the dot- and cross-product closed forms for 1 x 1, the normalisation and
  sign readings, and path/nnz counts from the selection rule.
"""

import os
from fractions import Fraction
from math import factorial, sqrt

import numpy as np
import pytest

from oracle import cg, irreps, sh, wigner
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
L_MAX_TEST = 3


def _triples(lmax=L_MAX_TEST):
    for l1 in range(lmax + 1):
        for l2 in range(lmax + 1):
            for l3 in range(abs(l1 - l2), l1 + l2 + 1):
                yield l1, l2, l3


def test_complex_orthogonality_both_directions():
    for l1 in range(L_MAX_TEST + 1):
        for l2 in range(L_MAX_TEST + 1):
            # rows: (m1, m2); columns: (l3, m3) over every allowed l3 -> square orthogonal matrix
            cols = []
            for l3 in range(abs(l1 - l2), l1 + l2 + 1):
                blk = cg.cg_complex_block(l1, l2, l3)
                cols.append(blk.reshape(-1, 2 * l3 + 1))
            u = np.concatenate(cols, axis=1)
            assert u.shape[0] == u.shape[1]
            np.testing.assert_allclose(u.T @ u, np.eye(u.shape[0]), atol=1e-13)
            np.testing.assert_allclose(u @ u.T, np.eye(u.shape[0]), atol=1e-13)


def test_complex_golden_table():
    path = os.path.join(GOLDEN, "cg_condon_shortley.txt")
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    assert len(rows) >= 20
    for l1, m1, l2, m2, big_l, big_m, sign, num, den in rows:
        expect = int(sign) * sqrt(int(num) / int(den))
        got = cg.cg_complex(int(l1), int(m1), int(l2), int(m2), int(big_l), int(big_m))
        assert abs(got - expect) < 1e-14, (l1, m1, l2, m2, big_l, big_m, got, expect)


def test_complex_closed_forms():
    f = factorial
    for l1 in range(5):
        for l2 in range(5):
            # L = 0: delta_{l1 l2} delta_{m1,-m2} (-1)^{l1-m1} / sqrt(2 l1 + 1)
            for m1 in range(-l1, l1 + 1):
                m2 = -m1
                if abs(m2) <= l2:
                    expect = (-1) ** (l1 - m1) / sqrt(2 * l1 + 1) if l1 == l2 else 0.0
                    assert abs(cg.cg_complex(l1, m1, l2, m2, 0, 0) - expect) < 1e-14
            # stretched L = l1 + l2
            big_l = l1 + l2
            for m1 in range(-l1, l1 + 1):
                for m2 in range(-l2, l2 + 1):
                    m = m1 + m2
                    expect = sqrt(Fraction(f(2 * l1) * f(2 * l2), f(2 * big_l))
                                  * Fraction(f(big_l + m) * f(big_l - m),
                                             f(l1 + m1) * f(l1 - m1) * f(l2 + m2) * f(l2 - m2)))
                    assert abs(cg.cg_complex(l1, m1, l2, m2, big_l, m) - expect) < 1e-13
        # coupling with l2 = 0 is the identity
        for m in range(-l1, l1 + 1):
            assert abs(cg.cg_complex(l1, m, 0, 0, l1, m) - 1.0) < 1e-14


def test_complex_against_sympy():
    sympy_cg = pytest.importorskip("sympy.physics.quantum.cg")
    for l1, l2, l3 in _triples(3):
        for m1 in range(-l1, l1 + 1):
            for m2 in range(-l2, l2 + 1):
                m3 = m1 + m2
                if abs(m3) > l3:
                    continue
                ref = float(sympy_cg.CG(l1, m1, l2, m2, l3, m3).doit())
                assert abs(cg.cg_complex(l1, m1, l2, m2, l3, m3) - ref) < 1e-13


def test_basis_change_is_unitary():
    for l in range(5):
        q = cg.real_basis_change(l)
        np.testing.assert_allclose(q @ q.conj().T, np.eye(2 * l + 1), atol=1e-15)


@pytest.mark.parametrize("seed", [0, 1])
def test_real_equivariance(seed):
    rng = np.random.default_rng(seed)
    rot = wigner.random_rotation(rng)
    d = [wigner.wigner_d_real(l, rot) for l in range(2 * L_MAX_TEST + 1)]
    for l1, l2, l3 in _triples():
        c = cg.cg_real_block(l1, l2, l3)
        lhs = np.einsum("abc,ai,bj->ijc", c, d[l1], d[l2])  # C(D1 e_i, D2 e_j)
        rhs = np.einsum("kc,ijc->ijk", d[l3], c)                 # D3 C(e_i, e_j)
        np.testing.assert_allclose(lhs, rhs, atol=1e-10, err_msg=str((l1, l2, l3)))


def test_real_normalisation_and_sign_rule():
    for l1, l2, l3 in _triples():
        c = cg.cg_real_block(l1, l2, l3)
        gram = np.einsum("abc,abd->cd", c, c)
        np.testing.assert_allclose(gram, np.eye(2 * l3 + 1), atol=1e-13)
        flat = c.reshape(-1)
        assert flat[np.nonzero(flat)[0][0]] > 0


def test_real_even_triples_match_gaunt_quadrature():
    # For l1 + l2 + l3 even the real coupling tensor is proportional to the
    # integral of a product of three real harmonics over the sphere.
    nodes, weights = np.polynomial.legendre.leggauss(24)
    n_phi = 48
    phi = (np.arange(n_phi) + 0.5) * 2 * np.pi / n_phi
    ct, ph = np.meshgrid(nodes, phi, indexing="ij")
    st = np.sqrt(1 - ct * ct)
    pts = np.stack([st * np.cos(ph), st * np.sin(ph), ct], axis=-1).reshape(-1, 3)
    wts = (weights[:, None] * np.full(n_phi, 2 * np.pi / n_phi)[None, :]).reshape(-1)
    ys = [sh.sh_real(l, pts) for l in range(2 * L_MAX_TEST + 1)]
    checked = 0
    for l1, l2, l3 in _triples():
        if (l1 + l2 + l3) % 2:
            continue
        gaunt = np.einsum("p,pa,pb,pc->abc", wts, ys[l1], ys[l2], ys[l3])
        gaunt *= sqrt((2 * l3 + 1) / np.sum(gaunt * gaunt))
        flat = gaunt.reshape(-1)
        if flat[np.abs(flat) > 1e-9][0] < 0:
            gaunt = -gaunt
        np.testing.assert_allclose(cg.cg_real_block(l1, l2, l3), gaunt, atol=1e-10)
        checked += 1
    assert checked >= 20


def test_real_closed_forms_1x1():
    s = 1 / sqrt(3)
    np.testing.assert_allclose(cg.cg_real_block(1, 1, 0)[:, :, 0], s * np.eye(3), atol=1e-15)
    # (y, z, x) basis: the 1 x 1 -> 1 block is the cross product / sqrt 2
    eps = np.zeros((3, 3, 3))
    yzx = {0: 1, 1: 2, 2: 0}  # component index -> Cartesian axis (x=0, y=1, z=2)
    for a in range(3):
        for b in range(3):
            for c_ in range(3):
                ia, ib, ic = yzx[a], yzx[b], yzx[c_]
                eps[a, b, c_] = np.linalg.det(np.eye(3)[[ia, ib, ic]])
    np.testing.assert_allclose(cg.cg_real_block(1, 1, 1), eps / sqrt(2), atol=1e-15)
    c2 = cg.cg_real_block(1, 1, 2)
    assert abs(c2[0, 0, 2] - 1 / sqrt(6)) < 1e-15       # (y, y) -> m = 0
    assert abs(c2[1, 1, 2] + 2 / sqrt(6)) < 1e-15       # (z, z) -> m = 0
    assert abs(abs(c2[0, 2, 0]) - 1 / sqrt(2)) < 1e-15  # (y, x) -> m = -2 (xy)
    # identity couplings with a scalar
    for l in range(4):
        np.testing.assert_allclose(cg.cg_real_block(l, 0, l)[:, 0, :], np.eye(2 * l + 1), atol=1e-14)
        np.testing.assert_allclose(cg.cg_real_block(0, l, l)[0], np.eye(2 * l + 1), atol=1e-14)


def test_paths_and_counts():
    # tiny: lmax 1, natural parity; derived by hand from the selection rule
    assert irreps.paths(1, False) == [(0, 0, 0), (0, 1, 1), (1, 0, 1), (1, 1, 0)]
    assert [irreps.irrep_name(i) for i in irreps.x_irreps(2, True)] == ["0e", "0o", "1o", "1e", "2e", "2o"]
    assert [irreps.irrep_name(i) for i in irreps.env_irreps(3)] == ["0e", "1o", "2e", "3o"]
    for lmax in (1, 2, 3):
        for full in (False, True):
            d1, d2, n_paths = workloads.dims(lmax, full)
            ps = irreps.paths(lmax, full)
            assert len(ps) == n_paths
            assert irreps.dim(irreps.x_irreps(lmax, full)) == d1
            assert irreps.dim(irreps.env_irreps(lmax)) == d2
            xs, es = irreps.x_irreps(lmax, full), irreps.env_irreps(lmax)
            for a, b, c in ps:
                assert xs[c][1] == xs[a][1] * es[b][1]
            assert ps == sorted(ps)
    # number of non-zeros of the combined tensor: invariant counts for lmax 2 / 3 full parity
    assert len(cg.combined_sparse(2, True)) == 274
    assert len(cg.combined_sparse(3, True)) == 1222
    assert len(cg.combined_sparse(1, False)) == 10
