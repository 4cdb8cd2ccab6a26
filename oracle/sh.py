"""Real spherical harmonics of edge directions (oracle, test infrastructure).

The paper embeds edge vectors into a spherical-harmonics basis in fp64 and
casts the result to fp32 (Appendix, "Mixed-Precision Architecture").  Here the
harmonics are built from their definition:

  * complex harmonics with the Condon-Shortley phase,
        Y_l^m = sqrt((2l+1)/(4 pi) (l-m)!/(l+m)!) P_l^m(cos theta) e^{i m phi},  m >= 0,
        Y_l^{-m} = (-1)^m conj(Y_l^m),
    with the associated Legendre functions P_l^m from the standard three-term
    recurrence in l.  P_l^m(z) carries a factor (1 - z^2)^{m/2}, and
    (1 - z^2)^{m/2} e^{i m phi} = (x + i y)^m on the unit sphere, so the
    "reduced" polynomial part is recurred and multiplied by (x + i y)^m;
  * the real harmonics Y^R = Q_l Y^C with Q_l from ``cg.real_basis_change``;
  * "component" normalisation (a reading; the paper does not state one):
    sum_m (Y_l^m)^2 = 2l + 1 on the unit sphere, i.e. the orthonormal
    harmonics times sqrt(4 pi), so Y_0 = 1 and Y_1 = sqrt(3) (y, z, x).

Parity unpinned for the normalisation and sign conventions (readings); the
values themselves are pinned by the Cartesian closed forms, scipy's complex
harmonics, the addition theorem and quadrature orthonormality.  The gradient
with respect to the edge vector is exact (the derivative of the same
recurrence); it is pinned by finite differences of the values, closed forms
for l = 1 and 2, homogeneity and rotation equivariance, and its VJP by
directional differences of the loss <grad_Y, Y(r)>.
"""

from __future__ import annotations

from math import factorial, pi, sqrt

import numpy as np

from .cg import real_basis_change


def _unit(xyz) -> np.ndarray:
    v = np.asarray(xyz, dtype=np.float64)
    return v / np.linalg.norm(v, axis=-1, keepdims=True)


def _reduced_legendre(l: int, m: int, z):
    """R_l^m(z) and its derivative dR_l^m/dz, for 0 <= m <= l.

    P_l^m(z) = (1 - z^2)^{m/2} R_l^m(z) with the Condon-Shortley phase:
        R_m^m = (-1)^m (2m - 1)!!,   R_{m+1}^m = (2m + 1) z R_m^m,
        (k - m) R_k^m = (2k - 1) z R_{k-1}^m - (k + m - 1) R_{k-2}^m.
    The derivative follows the same recurrence differentiated term by term:
        dR_m^m = 0,   dR_{m+1}^m = (2m + 1) R_m^m,
        (k - m) dR_k^m = (2k - 1) (R_{k-1}^m + z dR_{k-1}^m) - (k + m - 1) dR_{k-2}^m.
    """
    double_fact = 1.0
    for t in range(1, 2 * m, 2):
        double_fact *= t
    r_prev = np.full(np.shape(z), (-1.0) ** m * double_fact)
    d_prev = np.zeros(np.shape(z))
    if l == m:
        return r_prev, d_prev
    r_cur, d_cur = z * (2 * m + 1) * r_prev, (2 * m + 1) * r_prev
    for k in range(m + 2, l + 1):
        r_next = ((2 * k - 1) * z * r_cur - (k + m - 1) * r_prev) / (k - m)
        d_next = ((2 * k - 1) * (r_cur + z * d_cur) - (k + m - 1) * d_prev) / (k - m)
        r_prev, r_cur, d_prev, d_cur = r_cur, r_next, d_cur, d_next
    return r_cur, d_cur


def _norm(l: int, m: int) -> float:
    return sqrt((2 * l + 1) / (4 * pi) * factorial(l - m) / factorial(l + m))


def sh_complex(l: int, xyz) -> np.ndarray:
    """Orthonormal complex harmonics [n, 2l+1] (m = -l..l) at the directions xyz [n, 3]."""
    v = _unit(xyz)
    x, y, z = v[..., 0], v[..., 1], v[..., 2]
    n = v.shape[:-1]
    out = np.zeros(n + (2 * l + 1,), dtype=complex)
    for m in range(0, l + 1):
        r_l, _ = _reduced_legendre(l, m, z)
        ym = _norm(l, m) * r_l * (x + 1j * y) ** m
        out[..., l + m] = ym
        if m > 0:
            out[..., l - m] = (-1) ** m * np.conj(ym)
    return out


def sh_complex_grad_u(l: int, u) -> np.ndarray:
    """Gradient of the complex harmonics' polynomial form in the unit vector, [n, 2l+1, 3].

    For m >= 0, Y_l^m = N R_l^m(u_z) (u_x + i u_y)^m is a polynomial in the
    components of u; its partial derivatives (the components taken as
    independent variables) are
        d/du_x = N R (m (u_x + i u_y)^{m-1}),  d/du_y = i d/du_x,
        d/du_z = N (dR/dz) (u_x + i u_y)^m,
    and Y_l^{-m} = (-1)^m conj(Y_l^m) gives the negative orders.  Only the part
    tangent to the sphere survives the chain rule through u = r/|r|.
    """
    v = np.asarray(u, dtype=np.float64)
    x, y, z = v[..., 0], v[..., 1], v[..., 2]
    out = np.zeros(v.shape[:-1] + (2 * l + 1, 3), dtype=complex)
    w = x + 1j * y
    for m in range(0, l + 1):
        r_l, dr_l = _reduced_legendre(l, m, z)
        nm = _norm(l, m)
        dw = m * w ** (m - 1) if m > 0 else np.zeros_like(w)
        col = np.stack([nm * r_l * dw, 1j * nm * r_l * dw, nm * dr_l * w ** m], axis=-1)
        out[..., l + m, :] = col
        if m > 0:
            out[..., l - m, :] = (-1) ** m * np.conj(col)
    return out


def sh_real(l: int, xyz) -> np.ndarray:
    """Real harmonics of order l, component normalisation, shape [n, 2l+1]."""
    yc = sh_complex(l, xyz)
    yr = yc @ real_basis_change(l).T
    assert np.abs(yr.imag).max(initial=0.0) < 1e-12
    return yr.real * sqrt(4 * pi)


def sh_real_all(lmax: int, xyz) -> np.ndarray:
    """Concatenated real harmonics for l = 0..lmax, shape [n, (lmax+1)^2]."""
    return np.concatenate([sh_real(l, xyz) for l in range(lmax + 1)], axis=-1)


def sh_real_all_grad(lmax: int, vec) -> np.ndarray:
    """d Y_j / d vec for the concatenated real harmonics, shape [n, (lmax+1)^2, 3].

    Y depends on the direction only (Y(s r) = Y(r) for s > 0) and is evaluated
    on the edge vector r_ij itself, so this is the gradient with respect to the
    edge vector.  Exact (fp64): the gradient of the polynomial form in the unit
    vector (``sh_complex_grad_u``, from the derivative of the Legendre
    recurrence and the product rule on (u_x + i u_y)^m), chained through
    du/dr = (I - u u^T)/|r|, then moved to the real basis by the same Q_l and
    scaled like the values (component normalisation).
    """
    v = np.asarray(vec, dtype=np.float64)
    r = np.linalg.norm(v, axis=-1)
    u = v / r[..., None]
    proj = (np.eye(3) - u[..., :, None] * u[..., None, :]) / r[..., None, None]
    blocks = []
    for l in range(lmax + 1):
        jc = np.einsum("...mk,...kq->...mq", sh_complex_grad_u(l, u), proj)
        jr = np.einsum("am,...mq->...aq", real_basis_change(l), jc)
        assert np.abs(jr.imag).max(initial=0.0) < 1e-10 * max(1.0, np.abs(jr.real).max(initial=0.0))
        blocks.append(jr.real * sqrt(4 * pi))
    return np.concatenate(blocks, axis=-2)


def sh_backward(lmax: int, vec, grad_y) -> np.ndarray:
    """VJP of the harmonics: grad_vec[e] = sum_j grad_Y[e, j] dY_j/d vec_e (fp64)."""
    return np.einsum("ej,ejk->ek", np.asarray(grad_y, dtype=np.float64), sh_real_all_grad(lmax, vec))
