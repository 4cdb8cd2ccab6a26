"""Parity metric shared by the GPU tests.

err = max over elements of |got - ref| / max(|ref|, rms_blk(ref)), where
rms_blk is the RMS of the reference over the same irrep block (all edges and
channels).  A plain elementwise relative error is meaningless near the
cancellation zeros of a tensor product; the block RMS gives the natural scale
of every component.  Bars: 1e-5 for the forward (env, out), 1e-4 for the
backward (grad_x, grad_env, grad_w, grad_Y).
"""

import numpy as np

FWD_TOL = 1e-5
BWD_TOL = 1e-4


def block_rel_err(got, ref, blocks=None) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    blocks = blocks if blocks is not None else [slice(None)]
    err = 0.0
    for sl in blocks:
        o, g = ref[..., sl], got[..., sl]
        if o.size == 0:
            continue
        rms = float(np.sqrt(np.mean(o * o)))
        den = np.maximum(np.abs(o), rms)
        den = np.where(den == 0, 1.0, den)
        err = max(err, float(np.max(np.abs(g - o) / den)))
    if not np.all(np.isfinite(got)):
        return float("inf")
    return err
