"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the bench.

This module holds no tensor-product or embedding arithmetic: it only draws
random numbers, builds neighbour lists and evaluates the spherical harmonics
of edge directions (input preparation that sits before the library, which
takes Y as an input).  The harmonics are written out as Cartesian polynomials,
independently of the oracle's Legendre recurrence.

Workloads stand in for the paper's liquid-water boxes (§III.C): uniform random
atoms at 0.1 atoms/A^3 (the number density of water at 1 g/cm^3) in a periodic
cube, edges to every neighbour closer than the cutoff, model shapes from
Table I (lmax 2 / 64 features and lmax 3 / 128 features).  The SPICE 2 and
water trajectories of the paper are not used.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from math import sqrt

import numpy as np

BASE_SEED = 20250422


@dataclass(frozen=True)
class Config:
    name: str
    index: int            # seed offset
    n_atoms: int
    box: float            # cube edge, A
    cutoff: float         # A, edges need |r| < cutoff strictly
    U: int                # channels ("tensor features")
    lmax: int
    full_parity: bool
    host_features: bool   # features drawn with numpy on the host (else torch on the device)
    extra: dict = field(default_factory=dict)


def _box(n_atoms: int, density: float = 0.1) -> float:
    return (n_atoms / density) ** (1.0 / 3.0)


CONFIGS = {
    "tiny": Config("tiny", 0, 64, 10.0, 4.0, 16, 1, False, True),
    "small": Config("small", 1, 1000, _box(1000), 5.0, 32, 2, True, True),
    "headline": Config("headline", 2, 20000, _box(20000), 5.0, 64, 2, True, False),
    "large": Config("large", 3, 100000, _box(100000), 6.0, 64, 2, True, False),
    "high_order": Config("high_order", 4, 20000, _box(20000), 5.0, 128, 3, True, False),
    # one Allegro layer at the medium model shape of Table I (lmax 3, 64 features),
    # latent width L and MLP hidden width H as stated (readings)
    "layer_small": Config("layer_small", 5, 100, _box(100), 4.5, 64, 3, True, True, {"L": 64, "H": 128}),
    "medium_layer": Config("medium_layer", 6, 20000, _box(20000), 5.0, 64, 3, True, False, {"L": 64, "H": 128}),
}


def seed_streams(index: int):
    """Five independent child seeds: positions, x, w, path weights, upstream gradient."""
    return np.random.SeedSequence(BASE_SEED + index).spawn(5)


# ----------------------------------------------------------------- geometry

def neighbor_list(pos: np.ndarray, box: float, cutoff: float):
    """Directed edges i -> j (both directions), |r_ij| < cutoff, minimum image.

    Returns (row_ptr [N+1] int64, nbr [E] int64, vec [E, 3] float64) sorted by
    (center i, neighbour j); r_ij = r_j - r_i.  Requires cutoff < box / 2.
    """
    from scipy.spatial import cKDTree

    if not cutoff < box / 2:
        raise ValueError("cutoff must be below half the box edge")
    n = len(pos)
    tree = cKDTree(pos, boxsize=box)
    pairs = tree.query_pairs(r=cutoff, output_type="ndarray").astype(np.int64)
    i, j = pairs[:, 0], pairs[:, 1]
    d = pos[j] - pos[i]
    d -= box * np.round(d / box)
    r = np.linalg.norm(d, axis=1)
    keep = (r < cutoff) & (r > 1e-6)
    i, j, d = i[keep], j[keep], d[keep]
    centers = np.concatenate([i, j])
    nbrs = np.concatenate([j, i])
    vecs = np.concatenate([d, -d])
    order = np.lexsort((nbrs, centers))
    centers, nbrs, vecs = centers[order], nbrs[order], vecs[order]
    row_ptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(np.bincount(centers, minlength=n), out=row_ptr[1:])
    return row_ptr, nbrs, vecs


def real_sh_cartesian(lmax: int, vec: np.ndarray) -> np.ndarray:
    """Real spherical harmonics, component normalisation (sum_m Y^2 = 2l+1), l <= 3.

    Columns: l = 0..lmax, m = -l..l.  Written as polynomials of the unit vector
    (x, y, z); Y_1 = sqrt(3) (y, z, x).
    """
    if lmax > 3:
        raise ValueError("lmax <= 3")
    v = np.asarray(vec, dtype=np.float64)
    v = v / np.linalg.norm(v, axis=1, keepdims=True)
    x, y, z = v[:, 0], v[:, 1], v[:, 2]
    cols = [np.ones_like(x)]
    if lmax >= 1:
        s3 = sqrt(3.0)
        cols += [s3 * y, s3 * z, s3 * x]
    if lmax >= 2:
        s15, s5 = sqrt(15.0), sqrt(5.0)
        cols += [s15 * x * y, s15 * y * z, 0.5 * s5 * (3 * z * z - 1), s15 * x * z, 0.5 * s15 * (x * x - y * y)]
    if lmax >= 3:
        c3, c2, c1, c0 = sqrt(70.0) / 4, sqrt(105.0), sqrt(42.0) / 4, sqrt(7.0) / 2
        cols += [c3 * y * (3 * x * x - y * y), c2 * x * y * z, c1 * y * (5 * z * z - 1), c0 * z * (5 * z * z - 3),
                 c1 * x * (5 * z * z - 1), 0.5 * c2 * z * (x * x - y * y), c3 * x * (x * x - 3 * y * y)]
    return np.stack(cols, axis=1)


def dims(lmax: int, full_parity: bool):
    """(d1, d2, n_paths) from the irrep and path rules (counted, not enumerated by the oracle)."""
    d1 = sum((2 * l + 1) * (2 if full_parity else 1) for l in range(lmax + 1))
    d2 = (lmax + 1) ** 2
    n_paths = 0
    for la in range(lmax + 1):
        for lb in range(lmax + 1):
            for lc in range(abs(la - lb), min(la + lb, lmax) + 1):
                # x parity pa, env parity (-1)^lb; output parity is then fixed.
                # natural-only: pa = (-1)^la, pc must be (-1)^lc
                if full_parity:
                    n_paths += 2
                elif (la + lb + lc) % 2 == 0:
                    n_paths += 1
    return d1, d2, n_paths


@dataclass
class Graph:
    config: Config
    pos: np.ndarray
    row_ptr: np.ndarray
    nbr: np.ndarray
    vec: np.ndarray
    Y: np.ndarray  # float32 [E, d2], computed in fp64 then cast

    @property
    def n_edges(self) -> int:
        return int(self.row_ptr[-1])

    @property
    def n_atoms(self) -> int:
        return len(self.row_ptr) - 1


def make_graph(name: str) -> Graph:
    cfg = CONFIGS[name]
    ss = seed_streams(cfg.index)
    rng = np.random.default_rng(ss[0])
    pos = rng.uniform(0.0, cfg.box, size=(cfg.n_atoms, 3))
    row_ptr, nbr, vec = neighbor_list(pos, cfg.box, cfg.cutoff)
    y = real_sh_cartesian(cfg.lmax, vec).astype(np.float32)
    return Graph(cfg, pos, row_ptr, nbr, vec, y)


def host_features(cfg: Config, n_edges: int):
    """(x [E,U,d1], w [E,U], path_w [P,U], g [E,U,d1]) float32 drawn with numpy."""
    d1, _, n_paths = dims(cfg.lmax, cfg.full_parity)
    ss = seed_streams(cfg.index)
    x = np.random.default_rng(ss[1]).standard_normal((n_edges, cfg.U, d1), dtype=np.float32)
    w = np.random.default_rng(ss[2]).standard_normal((n_edges, cfg.U), dtype=np.float32)
    path_w = path_weights(cfg)
    g = np.random.default_rng(ss[4]).standard_normal((n_edges, cfg.U, d1), dtype=np.float32)
    return x, w, path_w, g


def path_weights(cfg: Config) -> np.ndarray:
    """Per-path, per-channel weights ~ N(0, sd = 1/sqrt(n_paths)), float32 [P, U]."""
    _, _, n_paths = dims(cfg.lmax, cfg.full_parity)
    rng = np.random.default_rng(seed_streams(cfg.index)[3])
    return (rng.standard_normal((n_paths, cfg.U)) / sqrt(n_paths)).astype(np.float32)


def device_features(cfg: Config, n_edges: int, device):
    """(x, w, g) as float32 torch tensors drawn on the device; path_w from the host."""
    import torch

    d1, _, _ = dims(cfg.lmax, cfg.full_parity)
    ss = seed_streams(cfg.index)

    def gen(child):
        g = torch.Generator(device=device)
        g.manual_seed(int(child.generate_state(1, dtype=np.uint64)[0] & 0x7FFFFFFFFFFFFFFF))
        return g

    x = torch.randn((n_edges, cfg.U, d1), generator=gen(ss[1]), device=device, dtype=torch.float32)
    w = torch.randn((n_edges, cfg.U), generator=gen(ss[2]), device=device, dtype=torch.float32)
    g = torch.randn((n_edges, cfg.U, d1), generator=gen(ss[4]), device=device, dtype=torch.float32)
    return x, w, g


def segment_prefix(row_ptr: np.ndarray, max_edges: int) -> int:
    """Number of leading centers whose segments together hold at most max_edges edges (>= 1)."""
    n = int(np.searchsorted(row_ptr, max_edges, side="right")) - 1
    return max(1, min(n, len(row_ptr) - 1))


def layer_params(cfg: Config):
    """Weights of one layer, float32, scaled by 1/sqrt(fan-in):
    A [L, U], W [P, U], Mix [n_x_irreps, U, U], B1 [L + U, H], B2 [H, L]."""
    d1, _, n_paths = dims(cfg.lmax, cfg.full_parity)
    L, H, U = cfg.extra["L"], cfg.extra["H"], cfg.U
    n_x = 2 * (cfg.lmax + 1) if cfg.full_parity else cfg.lmax + 1
    rng = np.random.default_rng(seed_streams(cfg.index)[3])
    shapes = {"A": ((L, U), L), "Mix": ((n_x, U, U), U), "B1": ((L + U, H), L + U), "B2": ((H, L), H)}
    prm = {k: (rng.standard_normal(s) / sqrt(fan)).astype(np.float32) for k, (s, fan) in shapes.items()}
    prm["W"] = path_weights(cfg)
    return prm


def layer_inputs(cfg: Config, n_edges: int, device=None):
    """(h [E, L], V [E, U, d1], dh_out [E, L], dV_out [E, U, d1]) float32 ~ N(0, 1):
    numpy arrays, or torch tensors drawn on `device` when it is given."""
    d1, _, _ = dims(cfg.lmax, cfg.full_parity)
    L, U = cfg.extra["L"], cfg.U
    ss = seed_streams(cfg.index)
    shapes = [(ss[1], (n_edges, L)), (ss[2], (n_edges, U, d1)), (ss[4], (n_edges, L)), (ss[0], (n_edges, U, d1))]
    if device is None:
        return tuple(np.random.default_rng(np.random.SeedSequence(int(c.generate_state(1)[0]) + 17))
                     .standard_normal(shape, dtype=np.float32) for c, shape in shapes)
    import torch

    out = []
    for child, shape in shapes:
        g = torch.Generator(device=device)
        g.manual_seed(int(child.generate_state(2, dtype=np.uint64)[1] & 0x7FFFFFFFFFFFFFFF))
        out.append(torch.randn(shape, generator=g, device=device, dtype=torch.float32))
    return tuple(out)
