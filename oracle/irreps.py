"""Irreducible-representation lists and coupling paths (oracle, test infrastructure).

An irrep is written (l, p): rotation order l >= 0 and parity p = +1 ("e") or
-1 ("o").  Within an irrep block the components run m = -l .. l, and blocks
are concatenated along the feature axis.

Readings (the paper fixes model shapes, Table I, but not the irrep lists):
  * Edge features x and the tensor-product output use the same irreps: for
    l = 0 .. lmax first the natural parity (l, (-1)^l), then, with full parity,
    the other one (l, -(-1)^l).  "Natural parity only" keeps 0e, 1o, 2e, 3o.
  * The environment embedding is a weighted sum of spherical harmonics, so its
    irreps are those of Y^l: (l, (-1)^l) for l = 0 .. lmax.
  * A path (a, b, c) couples x-irrep a with env-irrep b into out-irrep c when
    |l_a - l_b| <= l_c <= l_a + l_b and p_c = p_a * p_b.  Paths are ordered
    lexicographically by (a, b, c) in the irrep orders above; the position in
    that order is the path index p of the per-path weights W[p, u].
"""

from __future__ import annotations


def parity_name(p: int) -> str:
    return "e" if p == 1 else "o"


def irrep_name(ir) -> str:
    return f"{ir[0]}{parity_name(ir[1])}"


def x_irreps(lmax: int, full_parity: bool):
    """Irreps of the edge features x_ij and of the tensor-product output."""
    out = []
    for l in range(lmax + 1):
        natural = 1 if l % 2 == 0 else -1
        out.append((l, natural))
        if full_parity:
            out.append((l, -natural))
    return out


def env_irreps(lmax: int):
    """Irreps of the environment embedding: those of the harmonics Y^l."""
    return [(l, 1 if l % 2 == 0 else -1) for l in range(lmax + 1)]


def dim(irreps) -> int:
    return sum(2 * l + 1 for l, _ in irreps)


def offsets(irreps):
    """Start of each irrep block along the concatenated feature axis."""
    off, acc = [], 0
    for l, _ in irreps:
        off.append(acc)
        acc += 2 * l + 1
    return off


def paths(lmax: int, full_parity: bool):
    """All allowed (a, b, c) index triples in path order.

    a indexes x_irreps, b indexes env_irreps, c indexes x_irreps (the output).
    """
    xs = x_irreps(lmax, full_parity)
    es = env_irreps(lmax)
    result = []
    for a, (la, pa) in enumerate(xs):
        for b, (lb, pb) in enumerate(es):
            for c, (lc, pc) in enumerate(xs):
                if abs(la - lb) <= lc <= la + lb and pc == pa * pb:
                    result.append((a, b, c))
    return result
