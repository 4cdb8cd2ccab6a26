"""Pins of the oracle's Allegro layer (the composition around the tensor product).

* SiLU and its derivative against closed values and central differences;
* special cases: identity mixing and B2 = 0 give V' = TP(V, env) and h' = h,
  and the scalar track sees exactly the 0e components of the tensor product;
* rotation (and inversion) equivariance of the whole layer: h' invariant,
  every block of V' rotated by its Wigner matrix;
* the VJP against central differences in fp64 through every input and weight.
"""

import numpy as np
import pytest

import workloads
from oracle import layer, sh, tp, wigner


def _setup(lmax=2, full=True, U=3, L=4, H=5, seed=0, rot=None, n_atoms=8, box=6.0, cutoff=2.9):
    rng = np.random.default_rng(seed)
    pos = rng.uniform(0, box, size=(n_atoms, 3))
    row_ptr, _, vec = workloads.neighbor_list(pos, box, cutoff)
    if rot is not None:
        vec = vec @ rot.T
    lay = layer.AllegroLayer(lmax, full, U, L, H)
    e = int(row_ptr[-1])
    h = rng.standard_normal((e, L))
    V = rng.standard_normal((e, U, lay.tp.d1))
    prm = {k: rng.standard_normal(s) / np.sqrt(s[-2] if len(s) > 1 else 1) for k, s in lay.param_shapes().items()}
    return lay, row_ptr, h, V, sh.sh_real_all(lmax, vec), prm


def test_silu():
    a = np.linspace(-6, 6, 49)
    assert layer.silu(np.array(0.0)) == 0.0 and layer.silu_grad(np.array(0.0)) == 0.5
    np.testing.assert_allclose(layer.silu(a), a * 0.5 * (1 + np.tanh(a / 2)), rtol=1e-14, atol=1e-15)
    fd = (layer.silu(a + 1e-6) - layer.silu(a - 1e-6)) / 2e-6
    np.testing.assert_allclose(layer.silu_grad(a), fd, rtol=1e-8, atol=1e-9)


def test_special_cases():
    lay, row_ptr, h, V, Y, prm = _setup(seed=1)
    prm = dict(prm)
    prm["Mix"] = np.stack([np.eye(lay.U)] * lay.n_irreps)
    prm["B2"] = np.zeros_like(prm["B2"])
    h_out, V_out, cache = lay.forward(row_ptr, h, V, Y, prm)
    env = tp.env_embed(row_ptr, h @ prm["A"], Y)
    T = lay.tp.forward(row_ptr, V, env, prm["W"])
    np.testing.assert_allclose(V_out, T, rtol=0, atol=0)
    np.testing.assert_array_equal(h_out, h)
    # the scalar track reads the 0e block, which is component 0
    assert lay.tp.x_slices[0] == slice(0, 1) and lay.tp.x_irreps[0] == (0, 1)
    np.testing.assert_array_equal(cache["s"], T[:, :, 0])


@pytest.mark.parametrize("improper", [False, True])
def test_equivariance(improper):
    rng = np.random.default_rng(7)
    rot = wigner.random_rotation(rng)
    if improper:
        rot = -rot
    lay, row_ptr, h, V, Y, prm = _setup(lmax=2, full=True, seed=2)
    _, _, _, _, Y_rot, _ = _setup(lmax=2, full=True, seed=2, rot=rot)
    dx = wigner.wigner_d_blocks(lay.tp.x_irreps, rot)
    h1, V1, _ = lay.forward(row_ptr, h, V, Y, prm)
    h2, V2, _ = lay.forward(row_ptr, h, V @ dx.T, Y_rot, prm)
    np.testing.assert_allclose(h2, h1, atol=1e-10 * np.abs(h1).max())
    np.testing.assert_allclose(V2, V1 @ dx.T, atol=1e-10 * np.abs(V1).max())


@pytest.mark.parametrize("lmax,full", [(1, False), (2, True)])
def test_backward_finite_differences(lmax, full):
    lay, row_ptr, h, V, Y, prm = _setup(lmax=lmax, full=full, seed=3)
    rng = np.random.default_rng(4)
    h_o, V_o, _ = lay.forward(row_ptr, h, V, Y, prm)
    dh_out, dV_out = rng.standard_normal(h_o.shape), rng.standard_normal(V_o.shape)
    grads = lay.backward(row_ptr, h, V, Y, prm, dh_out, dV_out)

    def loss(h_, V_, Y_, prm_):
        a, b, _ = lay.forward(row_ptr, h_, V_, Y_, prm_)
        return np.sum(dh_out * a) + np.sum(dV_out * b)

    eps = 1e-6
    inputs = {"h": h, "V": V, "Y": Y}
    for name in ("h", "V", "Y", "A", "W", "Mix", "B1", "B2"):
        base = inputs[name] if name in inputs else prm[name]
        d = rng.standard_normal(base.shape)

        def shifted(sign):
            ins = dict(inputs)
            p2 = dict(prm)
            if name in ins:
                ins[name] = base + sign * eps * d
            else:
                p2[name] = base + sign * eps * d
            return loss(ins["h"], ins["V"], ins["Y"], p2)

        fd = (shifted(1) - shifted(-1)) / (2 * eps)
        an = np.sum(grads[name] * d)
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (name, fd, an)
