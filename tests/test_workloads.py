"""Invariants of the seeded input generator (host side, no GPU)."""

import numpy as np

import workloads
from oracle import sh


def test_neighbor_list_invariants():
    g = workloads.make_graph("tiny")
    rp, nbr, vec = g.row_ptr, g.nbr, g.vec
    assert rp[0] == 0 and rp[-1] == len(nbr) and np.all(np.diff(rp) >= 0)
    centers = np.repeat(np.arange(len(rp) - 1), np.diff(rp))
    assert np.all(centers != nbr)                                    # no self edges
    r = np.linalg.norm(vec, axis=1)
    assert np.all(r < g.config.cutoff) and np.all(r > 1e-6)
    fwd = set(zip(centers.tolist(), nbr.tolist()))
    assert fwd == set(zip(nbr.tolist(), centers.tolist()))           # symmetric edge set
    key = centers * len(rp) + nbr
    assert np.all(np.diff(key) > 0)                                   # sorted by (center, neighbour)
    # minimum image vectors
    d = g.pos[nbr] - g.pos[centers]
    d -= g.config.box * np.round(d / g.config.box)
    np.testing.assert_allclose(vec, d, atol=1e-12)
    # brute force over all pairs
    n = len(g.pos)
    dd = g.pos[None, :, :] - g.pos[:, None, :]
    dd -= g.config.box * np.round(dd / g.config.box)
    rr = np.linalg.norm(dd, axis=2)
    brute = {(i, j) for i in range(n) for j in range(n) if i != j and rr[i, j] < g.config.cutoff}
    assert brute == fwd


def test_degree_statistics_small():
    g = workloads.make_graph("small")
    cfg = g.config
    lam = (cfg.n_atoms - 1) / cfg.box ** 3 * 4 / 3 * np.pi * cfg.cutoff ** 3
    deg = np.diff(g.row_ptr)
    assert abs(deg.mean() - lam) < 0.05 * lam
    assert abs(deg.var() - lam) < 0.25 * lam                          # Poisson: variance = mean


def test_cartesian_harmonics_match_oracle_recurrence():
    v = np.random.default_rng(1).standard_normal((200, 3))
    np.testing.assert_allclose(workloads.real_sh_cartesian(3, v), sh.sh_real_all(3, v), atol=1e-13)


def test_seeded_features_reproducible():
    cfg = workloads.CONFIGS["tiny"]
    a = workloads.host_features(cfg, 100)
    b = workloads.host_features(cfg, 100)
    for u, v in zip(a, b):
        assert u.dtype == np.float32 and np.array_equal(u, v)
    x, w, path_w, g = a
    assert x.shape == (100, 16, 4) and w.shape == (100, 16) and path_w.shape == (4, 16) and g.shape == x.shape
    assert abs(path_w.std() - 0.5) < 0.2                              # sd = 1/sqrt(n_paths) = 0.5
