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
harmonics, the addition theorem and quadrature orthonormality.
"""

from __future__ import annotations

from math import factorial, pi, sqrt

import numpy as np

from .cg import real_basis_change


def _unit(xyz) -> np.ndarray:
    v = np.asarray(xyz, dtype=np.float64)
    return v / np.linalg.norm(v, axis=-1, keepdims=True)


def sh_complex(l: int, xyz) -> np.ndarray:
    """Orthonormal complex harmonics [n, 2l+1] (m = -l..l) at the directions xyz [n, 3]."""
    v = _unit(xyz)
    x, y, z = v[..., 0], v[..., 1], v[..., 2]
    n = v.shape[:-1]
    out = np.zeros(n + (2 * l + 1,), dtype=complex)
    for m in range(0, l + 1):
        # reduced associated Legendre R_k^m(z), P_k^m = (1-z^2)^{m/2} R_k^m, CS phase included
        double_fact = 1.0
        for t in range(1, 2 * m, 2):
            double_fact *= t
        r_prev = np.full(n, (-1.0) ** m * double_fact)  # R_m^m
        if l == m:
            r_l = r_prev
        else:
            r_cur = z * (2 * m + 1) * r_prev  # R_{m+1}^m
            for k in range(m + 2, l + 1):
                r_prev, r_cur = r_cur, ((2 * k - 1) * z * r_cur - (k + m - 1) * r_prev) / (k - m)
            r_l = r_cur
        norm = sqrt((2 * l + 1) / (4 * pi) * factorial(l - m) / factorial(l + m))
        ym = norm * r_l * (x + 1j * y) ** m
        out[..., l + m] = ym
        if m > 0:
            out[..., l - m] = (-1) ** m * np.conj(ym)
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


def sh_real_all_grad(lmax: int, vec, h: float = 1e-4) -> np.ndarray:
    """d Y_j / d vec for the concatenated real harmonics, shape [n, (lmax+1)^2, 3].

    Y depends on the direction only (Y(s r) = Y(r) for s > 0), and is evaluated
    on the vector itself (not its unit vector), so this is the gradient with
    respect to the edge vector r_ij.  Fourth-order central differences in fp64,
    with the step scaled by |r|:
        f'(r) = (-f(r + 2h) + 8 f(r + h) - 8 f(r - h) + f(r - 2h)) / (12 h).
    Truncation error O(h^4) and rounding O(eps / h) are both far below 1e-9
    relative for |r| of order 1.
    """
    v = np.asarray(vec, dtype=np.float64)
    scale = np.linalg.norm(v, axis=-1, keepdims=True)
    out = np.zeros(v.shape[:-1] + ((lmax + 1) ** 2, 3))
    for k in range(3):
        step = np.zeros_like(v)
        step[..., k] = h * scale[..., 0]
        f = [sh_real_all(lmax, v + c * step) for c in (2, 1, -1, -2)]
        out[..., k] = (-f[0] + 8 * f[1] - 8 * f[2] + f[3]) / (12 * h * scale)
    return out


def sh_backward(lmax: int, vec, grad_y) -> np.ndarray:
    """VJP of the harmonics: grad_vec[e] = sum_j grad_Y[e, j] dY_j/d vec_e (fp64)."""
    return np.einsum("ej,ejk->ek", np.asarray(grad_y, dtype=np.float64), sh_real_all_grad(lmax, vec))
