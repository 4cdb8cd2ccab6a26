"""One Allegro layer around the tensor product (oracle, test infrastructure).

The paper names the layer's parts but does not write them out: Allegro layers
mix equivariant tensor features with Clebsch-Gordan tensor products and update
scalar features with MLPs, in fp32 (Appendix, "Mixed-Precision Architecture";
Table I gives the model shapes; the layer itself is defined in the Allegro
papers it cites).  The composition below is a reading of that architecture,
written from its published description, with the tensor product of §II.D at
its center.  Per edge e (center c(e)), with scalar latent h [E, L], tensor
features V [E, U, d1] and edge harmonics Y [E, d2]:

  1. environment weights       w = h A                      A [L, U]
  2. environment embedding      env = env_embed(w, Y)        (segment sum)
  3. tensor product             T = TP(V, env; W)            W [P, U]
  4. per-irrep channel mixing   V'[e, u', k] = sum_u Mix[c(k), u', u] T[e, u, k]
                                (one U x U matrix per x irrep c)
  5. invariant scalars          s[e, u] = T[e, u, 0]         (the 0e component)
  6. latent update              a = [h, s] B1,  z = SiLU(a),  h' = h + z B2
                                B1 [L + U, H], B2 [H, L], SiLU(a) = a / (1 + exp(-a))

Outputs (h', V').  `backward` returns the VJP with respect to every input and
weight, written out step by step in reverse.  Everything is fp64 on the given
values.  Parity unpinned for the composition itself (a reading); each function
is pinned by finite differences, rotation equivariance and its special cases.
"""

from __future__ import annotations

import numpy as np

from . import tp as _tp


def silu(a):
    return a / (1.0 + np.exp(-a))


def silu_grad(a):
    sg = 1.0 / (1.0 + np.exp(-a))
    return sg * (1.0 + a * (1.0 - sg))


class AllegroLayer:
    """Shapes of one layer: (lmax, parity) of the tensor product, U channels, latent L, hidden H."""

    def __init__(self, lmax: int, full_parity: bool, U: int, L: int, H: int):
        self.tp = _tp.TensorProduct(lmax, full_parity)
        self.U, self.L, self.H = U, L, H
        # x irrep of every component k (the mixing matrix that acts on it)
        self.irrep_of = np.zeros(self.tp.d1, dtype=np.int64)
        for c, sl in enumerate(self.tp.x_slices):
            self.irrep_of[sl] = c
        self.n_irreps = len(self.tp.x_slices)

    def param_shapes(self):
        t = self.tp
        return {"A": (self.L, self.U), "W": (t.n_paths, self.U), "Mix": (self.n_irreps, self.U, self.U),
                "B1": (self.L + self.U, self.H), "B2": (self.H, self.L)}

    def mix(self, Mix, T):
        """V'[e, u', k] = sum_u Mix[c(k), u', u] T[e, u, k]."""
        out = np.zeros_like(T)
        for c, sl in enumerate(self.tp.x_slices):
            out[:, :, sl] = np.einsum("vu,euk->evk", Mix[c], T[:, :, sl])
        return out

    def forward(self, row_ptr, h, V, Y, prm):
        h, V, Y = (np.asarray(a, np.float64) for a in (h, V, Y))
        p = {k: np.asarray(v, np.float64) for k, v in prm.items()}
        w = h @ p["A"]
        env = _tp.env_embed(row_ptr, w, Y)
        T = self.tp.forward(row_ptr, V, env, p["W"])
        V_out = self.mix(p["Mix"], T)
        s = T[:, :, 0]
        a = np.concatenate([h, s], axis=1) @ p["B1"]
        z = silu(a)
        h_out = h + z @ p["B2"]
        cache = {"w": w, "env": env, "T": T, "s": s, "a": a, "z": z}
        return h_out, V_out, cache

    def backward(self, row_ptr, h, V, Y, prm, dh_out, dV_out):
        """Gradients of <dh_out, h'> + <dV_out, V'> with respect to h, V, Y and every weight."""
        h, V, Y = (np.asarray(a, np.float64) for a in (h, V, Y))
        p = {k: np.asarray(v, np.float64) for k, v in prm.items()}
        dh_out, dV_out = np.asarray(dh_out, np.float64), np.asarray(dV_out, np.float64)
        _, _, cch = self.forward(row_ptr, h, V, Y, prm)
        L = self.L
        hs = np.concatenate([h, cch["s"]], axis=1)
        # 6. latent update
        dB2 = cch["z"].T @ dh_out
        da = (dh_out @ p["B2"].T) * silu_grad(cch["a"])
        dB1 = hs.T @ da
        dhs = da @ p["B1"].T
        dh = dh_out + dhs[:, :L]
        # 4-5. mixing and the scalar read-out, back into T
        dT = np.zeros_like(cch["T"])
        dMix = np.zeros_like(p["Mix"])
        for c, sl in enumerate(self.tp.x_slices):
            dT[:, :, sl] = np.einsum("vu,evk->euk", p["Mix"][c], dV_out[:, :, sl])
            dMix[c] = np.einsum("evk,euk->vu", dV_out[:, :, sl], cch["T"][:, :, sl])
        dT[:, :, 0] += dhs[:, L:]
        # 3-2. tensor product and embedding
        dV, _, dw, dY = self.tp.backward(row_ptr, V, cch["env"], p["W"], dT, cch["w"], Y)
        dW = self.tp.path_weight_grad(row_ptr, V, cch["env"], dT)
        # 1. environment weights
        dA = h.T @ dw
        dh = dh + dw @ p["A"].T
        return {"h": dh, "V": dV, "Y": dY, "A": dA, "W": dW, "Mix": dMix, "B1": dB1, "B2": dB2}
