"""Clebsch-Gordan coupling tensors in the real basis (oracle, test infrastructure).

The paper's kernel stores "the combined tensor of Wigner 3-j contraction
coefficients" in a compressed sparse format (§II.D, last paragraph).  This
module builds that tensor from its textbook definition:

  1. complex Clebsch-Gordan coefficients <l1 m1 l2 m2 | l3 m3> in the
     Condon-Shortley convention, from Racah's closed formula evaluated exactly
     in rational arithmetic (one floating-point square root at the end);
  2. the change of basis Q_l from complex to real spherical-harmonic
     components (the same Q_l defines the real harmonics in ``sh.py``);
  3. the real coupling tensor
        C[a, b, c] = sum_{ijk} conj(Q_l1)[a, i] conj(Q_l2)[b, j] Q_l3[c, k] CG[i, j, k],
     which is purely real when l1+l2+l3 is even and purely imaginary when it is
     odd; the non-zero part is kept;
  4. the normalisation / sign reading (the paper is silent on both):
     sum_{m1,m2} C[m1,m2,m3] C[m1,m2,m3'] = delta_{m3 m3'} (so sum C^2 = 2 l3 + 1),
     and the first non-zero entry in row-major (m1, m2, m3) order is positive.

Parity unpinned: the sign rule and the overall scale are conventions; every
equivariance and orthogonality pin holds for any consistent choice.
"""

from __future__ import annotations

from fractions import Fraction
from functools import lru_cache
from math import factorial, sqrt

import numpy as np

from . import irreps as _irreps


@lru_cache(maxsize=None)
def cg_complex(l1: int, m1: int, l2: int, m2: int, l3: int, m3: int) -> float:
    """<l1 m1 l2 m2 | l3 m3>, Condon-Shortley phase, by Racah's formula.

    The squared prefactor and the alternating sum are exact rationals; only
    the final square root is floating point (fp64).
    """
    if m3 != m1 + m2:
        return 0.0
    if not abs(l1 - l2) <= l3 <= l1 + l2:
        return 0.0
    if abs(m1) > l1 or abs(m2) > l2 or abs(m3) > l3:
        return 0.0
    f = factorial
    pref_sq = Fraction(
        (2 * l3 + 1) * f(l3 + l1 - l2) * f(l3 - l1 + l2) * f(l1 + l2 - l3),
        f(l1 + l2 + l3 + 1),
    )
    pref_sq *= f(l3 + m3) * f(l3 - m3) * f(l1 - m1) * f(l1 + m1) * f(l2 - m2) * f(l2 + m2)
    s = Fraction(0)
    for k in range(l1 + l2 + l3 + 1):
        args = (k, l1 + l2 - l3 - k, l1 - m1 - k, l2 + m2 - k, l3 - l2 + m1 + k, l3 - l1 - m2 + k)
        if min(args) < 0:
            continue
        den = 1
        for v in args:
            den *= f(v)
        s += Fraction((-1) ** k, den)
    if s == 0:
        return 0.0
    mag = sqrt(pref_sq * s * s)
    return mag if s > 0 else -mag


def cg_complex_block(l1: int, l2: int, l3: int) -> np.ndarray:
    """Dense [2l1+1, 2l2+1, 2l3+1] array of complex-basis CG (real numbers)."""
    out = np.zeros((2 * l1 + 1, 2 * l2 + 1, 2 * l3 + 1))
    for i, m1 in enumerate(range(-l1, l1 + 1)):
        for j, m2 in enumerate(range(-l2, l2 + 1)):
            m3 = m1 + m2
            if abs(m3) <= l3:
                out[i, j, m3 + l3] = cg_complex(l1, m1, l2, m2, l3, m3)
    return out


def real_basis_change(l: int) -> np.ndarray:
    """Q_l: real components = Q_l @ complex components (row real m, column complex m').

    m > 0: Q[m, m] = (-1)^m / sqrt2,  Q[m, -m] = 1 / sqrt2
    m = 0: Q[0, 0] = 1
    m < 0: Q[m, m] = i / sqrt2,       Q[m, -m] = -i (-1)^m / sqrt2
    With Condon-Shortley harmonics this gives the textbook real harmonics with
    positive leading coefficients, e.g. l = 1 proportional to (y, z, x).
    Parity unpinned (a basis convention).
    """
    q = np.zeros((2 * l + 1, 2 * l + 1), dtype=complex)
    r2 = sqrt(2.0)
    for m in range(-l, l + 1):
        row = m + l
        if m > 0:
            q[row, m + l] = (-1) ** m / r2
            q[row, -m + l] = 1 / r2
        elif m == 0:
            q[row, l] = 1.0
        else:
            q[row, m + l] = 1j / r2
            q[row, -m + l] = -1j * (-1) ** m / r2
    return q


@lru_cache(maxsize=None)
def _real_block_cached(l1: int, l2: int, l3: int) -> np.ndarray:
    cg = cg_complex_block(l1, l2, l3)
    q1, q2, q3 = real_basis_change(l1), real_basis_change(l2), real_basis_change(l3)
    c = np.einsum("ai,bj,ck,ijk->abc", q1.conj(), q2.conj(), q3, cg)
    if (l1 + l2 + l3) % 2 == 0:
        assert np.abs(c.imag).max() < 1e-12, (l1, l2, l3)
        c = c.real.copy()
    else:
        assert np.abs(c.real).max() < 1e-12, (l1, l2, l3)
        c = c.imag.copy()
    # normalisation: orthonormal in (m1, m2) for each m3 -> total sum of squares 2 l3 + 1
    c *= sqrt((2 * l3 + 1) / float(np.sum(c * c)))
    # sign: first non-zero entry in row-major (m1, m2, m3) order is positive
    flat = c.reshape(-1)
    first = flat[np.abs(flat) > 1e-12 * np.abs(flat).max()][0]
    if first < 0:
        c = -c
    c[np.abs(c) < 1e-14] = 0.0
    c.setflags(write=False)
    return c


def cg_real_block(l1: int, l2: int, l3: int) -> np.ndarray:
    """Real coupling tensor C[m1, m2, m3] of shape [2l1+1, 2l2+1, 2l3+1] (a copy)."""
    if not abs(l1 - l2) <= l3 <= l1 + l2:
        raise ValueError("triangle rule violated")
    return _real_block_cached(l1, l2, l3).copy()


def coupling_tensors(lmax: int, full_parity: bool):
    """[(a, b, c, C_p)] for every path, in path order (see ``irreps.paths``)."""
    xs = _irreps.x_irreps(lmax, full_parity)
    es = _irreps.env_irreps(lmax)
    return [(a, b, c, cg_real_block(xs[a][0], es[b][0], xs[c][0]))
            for a, b, c in _irreps.paths(lmax, full_parity)]


def combined_sparse(lmax: int, full_parity: bool):
    """Compressed sparse combined coupling tensor (§II.D): list of (p, i, j, k, value).

    i indexes the concatenated x components, j the env components and k the
    output components; p is the path the entry belongs to.
    """
    xs = _irreps.x_irreps(lmax, full_parity)
    es = _irreps.env_irreps(lmax)
    xo, eo = _irreps.offsets(xs), _irreps.offsets(es)
    entries = []
    for p, (a, b, c, blk) in enumerate(coupling_tensors(lmax, full_parity)):
        for m1, m2, m3 in zip(*np.nonzero(blk)):
            entries.append((p, xo[a] + int(m1), eo[b] + int(m2), xo[c] + int(m3), float(blk[m1, m2, m3])))
    return entries
