"""Wigner-D matrices of the real harmonics basis (oracle test tool).

D^l(R) is defined by Y^l(R r) = D^l(R) Y^l(r) for every unit vector r.  It is
obtained by least squares from the harmonics at random directions, so it uses
no formula beyond the harmonics themselves.  Equivariance of the tensor
product (every output block rotates by D^{l3} when every input block rotates
by its own D) is the main pin of the coupling tensors.
"""

from __future__ import annotations

import numpy as np

from .sh import sh_real


def random_rotation(rng: np.random.Generator) -> np.ndarray:
    """Haar-random proper rotation (det +1) from the QR factors of a Gaussian matrix."""
    q, r = np.linalg.qr(rng.standard_normal((3, 3)))
    q = q @ np.diag(np.sign(np.diag(r)))
    if np.linalg.det(q) < 0:
        q[:, 0] = -q[:, 0]
    return q


def wigner_d_real(l: int, rot: np.ndarray, rng: np.random.Generator | None = None) -> np.ndarray:
    """[2l+1, 2l+1] matrix with sh_real(l, rot @ r) = D @ sh_real(l, r)."""
    rng = rng if rng is not None else np.random.default_rng(12345)
    pts = rng.standard_normal((8 * (2 * l + 1), 3))
    a = sh_real(l, pts)
    b = sh_real(l, pts @ rot.T)
    dt, *_ = np.linalg.lstsq(a, b, rcond=None)
    return dt.T


def wigner_d_blocks(irreps, rot: np.ndarray) -> np.ndarray:
    """Block-diagonal representation matrix for a concatenated irrep list.

    A proper rotation acts on block (l, p) by D^l; parity only enters under
    inversion (``rot`` with det -1), where block (l, p) picks up the factor p.
    """
    det = np.linalg.det(rot)
    proper = rot * np.sign(det)
    size = sum(2 * l + 1 for l, _ in irreps)
    out = np.zeros((size, size))
    off = 0
    for l, p in irreps:
        d = wigner_d_real(l, proper)
        if det < 0:
            d = d * p
        out[off:off + 2 * l + 1, off:off + 2 * l + 1] = d
        off += 2 * l + 1
    return out
