"""Environment embedding and the channel-wise tensor product, forward and VJP (oracle).

Test infrastructure only.  The paper names the Allegro tensor product as the
architecture's most expensive operation and implements it, and its first
derivative, as fused custom kernels (§II.D); its definition lives in the Allegro
papers the paper cites.  Restated (notation of the paper's model: edges ij with
center i, channels u, irreps (l, p)):

  environment embedding (a segment sum over the center-sorted edge list):
      env[n, u, j] = sum_{e in seg(n)} w[e, u] * Y[e, j]
  tensor product, channel-wise (channel u only meets channel u), one weight per
  path and channel:
      out[e, u, k] = sum_p W[p, u] sum_{(i, j, k) in p} C_ijk x[e, u, i] env[c(e), u, j]
  its VJP given g = dL/d out:
      grad_x[e, u, i]   = sum_p W[p, u] sum C_ijk env[c(e), u, j] g[e, u, k]
      grad_env[n, u, j] = sum_{e in seg(n)} sum_p W[p, u] sum C_ijk x[e, u, i] g[e, u, k]
  and the VJP of the embedding through grad_env:
      grad_w[e, u] = sum_j grad_env[c(e), u, j] Y[e, j]
      grad_Y[e, j] = sum_u grad_env[c(e), u, j] w[e, u]
  and, for training (the paper leaves its kernels to future work, §II.D), the
  gradient of the path weights, a reduction over every edge:
      grad_W[p, u] = sum_e sum_{(i, j, k) in p} C_ijk x[e, u, i] env[c(e), u, j] g[e, u, k]

Segments: edge e belongs to center n iff row_ptr[n] <= e < row_ptr[n+1]; an
empty segment gives env = 0 and grad_env = 0.

Precision (Appendix, "Mixed-Precision Architecture"): the GPU computes in fp32;
the oracle evaluates the definition in fp64 on the same fp32 input values.

Two forms: ``*_loops`` are plain nested Python loops (tiny inputs, brute force);
the default forms take the same steps per path over the dense coupling blocks,
in chunks of edges: the outer product of the two input blocks, flattened, times
the flattened block (a matmul).  Both must agree to fp64 rounding.
"""

from __future__ import annotations

import numpy as np

from . import cg as _cg
from . import irreps as _irreps

_CHUNK = 4096


def centers_of_edges(row_ptr) -> np.ndarray:
    """c(e) for every edge, from the CSR row pointer."""
    rp = np.asarray(row_ptr, dtype=np.int64)
    degrees = np.diff(rp)
    return np.repeat(np.arange(len(rp) - 1, dtype=np.int64), degrees)


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


# --------------------------------------------------------------------------- env

def _outer(xa, eb) -> np.ndarray:
    """[e * u, i * j] products x_i env_j (rows (e, u), columns i major)."""
    n = xa.shape[0] * xa.shape[1]
    return (xa[:, :, :, None] * eb[:, :, None, :]).reshape(n, -1)


def _flat(blk) -> np.ndarray:
    """Coupling block C[i, j, k] as a [(i, j), k] matrix, i major."""
    return blk.reshape(-1, blk.shape[2])


def env_embed(row_ptr, w, Y) -> np.ndarray:
    """env[n, u, j] = sum over the segment of n of w[e, u] Y[e, j], fp64."""
    rp = np.asarray(row_ptr, dtype=np.int64)
    w64, y64 = _f64(w), _f64(Y)
    n_centers = len(rp) - 1
    env = np.zeros((n_centers, w64.shape[1], y64.shape[1]))
    for n in range(n_centers):
        s, t = rp[n], rp[n + 1]
        if t > s:
            env[n] = w64[s:t].T @ y64[s:t]
    return env


def env_embed_loops(row_ptr, w, Y) -> np.ndarray:
    rp = [int(v) for v in row_ptr]
    w64, y64 = _f64(w), _f64(Y)
    n_centers, n_ch, d2 = len(rp) - 1, w64.shape[1], y64.shape[1]
    env = np.zeros((n_centers, n_ch, d2))
    for n in range(n_centers):
        for e in range(rp[n], rp[n + 1]):
            for u in range(n_ch):
                for j in range(d2):
                    env[n, u, j] += w64[e, u] * y64[e, j]
    return env


def env_embed_fp32_replay(row_ptr, w, Y) -> np.ndarray:
    """Deterministic-order fp32 reference (a reading of "bit-exact").

    env32 = 0; for e ascending within the segment:
        env32 = fl32(env32 + fl32(w[e, u] * Y[e, j]))
    i.e. one IEEE fp32 rounding after the product and one after the sum, no
    fused multiply-add.  Vectorised over (u, j), sequential over e.
    """
    rp = np.asarray(row_ptr, dtype=np.int64)
    w32 = np.asarray(w, dtype=np.float32)
    y32 = np.asarray(Y, dtype=np.float32)
    n_centers = len(rp) - 1
    env = np.zeros((n_centers, w32.shape[1], y32.shape[1]), dtype=np.float32)
    for n in range(n_centers):
        acc = np.zeros((w32.shape[1], y32.shape[1]), dtype=np.float32)
        for e in range(rp[n], rp[n + 1]):
            prod = np.multiply(w32[e][:, None], y32[e][None, :], dtype=np.float32)
            acc = np.add(acc, prod, dtype=np.float32)
        env[n] = acc
    return env


def env_embed_backward(row_ptr, grad_env, w, Y):
    """(grad_w [E, U], grad_Y [E, d2]) given grad_env [N, U, d2]."""
    c = centers_of_edges(row_ptr)
    ge = _f64(grad_env)[c]
    return np.einsum("euj,ej->eu", ge, _f64(Y)), np.einsum("euj,eu->ej", ge, _f64(w))


# --------------------------------------------------------------------------- TP

class TensorProduct:
    """The channel-wise tensor product for one (lmax, parity mode)."""

    def __init__(self, lmax: int, full_parity: bool):
        self.lmax = lmax
        self.full_parity = full_parity
        self.x_irreps = _irreps.x_irreps(lmax, full_parity)
        self.env_irreps = _irreps.env_irreps(lmax)
        self.d1 = _irreps.dim(self.x_irreps)
        self.d2 = _irreps.dim(self.env_irreps)
        self.paths = _irreps.paths(lmax, full_parity)
        self.blocks = [blk for *_, blk in _cg.coupling_tensors(lmax, full_parity)]
        xo, eo = _irreps.offsets(self.x_irreps), _irreps.offsets(self.env_irreps)
        self.x_slices = [slice(o, o + 2 * l + 1) for o, (l, _) in zip(xo, self.x_irreps)]
        self.env_slices = [slice(o, o + 2 * l + 1) for o, (l, _) in zip(eo, self.env_irreps)]

    def _groups(self):
        """Paths grouped by their input blocks (a, b), which share the products x_i env_j."""
        groups = {}
        for p, (a, b, _) in enumerate(self.paths):
            groups.setdefault((a, b), []).append(p)
        return groups.items()

    @property
    def n_paths(self) -> int:
        return len(self.paths)

    @property
    def nnz(self) -> int:
        return int(sum(np.count_nonzero(b) for b in self.blocks))

    # ---- forward
    def forward(self, row_ptr, x, env, W) -> np.ndarray:
        x64, env64, w64 = _f64(x), _f64(env), _f64(W)
        c = centers_of_edges(row_ptr)
        n_edges, n_ch, _ = x64.shape
        out = np.zeros((n_edges, n_ch, self.d1))
        for s in range(0, n_edges, _CHUNK):
            t = min(s + _CHUNK, n_edges)
            xe, ee = x64[s:t], env64[c[s:t]]
            for (a, b), group in self._groups():
                q = _outer(xe[:, :, self.x_slices[a]], ee[:, :, self.env_slices[b]])
                for p in group:
                    cc = self.paths[p][2]
                    contrib = (q @ _flat(self.blocks[p])).reshape(t - s, n_ch, -1)
                    out[s:t, :, self.x_slices[cc]] += w64[p][None, :, None] * contrib
        return out

    def forward_loops(self, row_ptr, x, env, W) -> np.ndarray:
        x64, env64, w64 = _f64(x), _f64(env), _f64(W)
        c = centers_of_edges(row_ptr)
        n_edges, n_ch, _ = x64.shape
        out = np.zeros((n_edges, n_ch, self.d1))
        for e in range(n_edges):
            n = c[e]
            for u in range(n_ch):
                for p, (a, b, cc) in enumerate(self.paths):
                    blk = self.blocks[p]
                    oa, ob, oc = self.x_slices[a].start, self.env_slices[b].start, self.x_slices[cc].start
                    for m1 in range(blk.shape[0]):
                        for m2 in range(blk.shape[1]):
                            for m3 in range(blk.shape[2]):
                                cv = blk[m1, m2, m3]
                                if cv != 0.0:
                                    out[e, u, oc + m3] += (w64[p, u] * cv * x64[e, u, oa + m1]
                                                           * env64[n, u, ob + m2])
        return out

    # ---- backward (VJP)
    def backward(self, row_ptr, x, env, W, g, w, Y):
        """(grad_x, grad_env, grad_w, grad_Y) for the upstream gradient g = dL/d out."""
        x64, env64, w64, g64 = _f64(x), _f64(env), _f64(W), _f64(g)
        c = centers_of_edges(row_ptr)
        n_edges, n_ch, _ = x64.shape
        grad_x = np.zeros_like(x64)
        grad_env_edge = np.zeros((n_edges, n_ch, self.d2))
        for s in range(0, n_edges, _CHUNK):
            t = min(s + _CHUNK, n_edges)
            xe, ee, ge = x64[s:t], env64[c[s:t]], g64[s:t]
            for p, (a, b, cc) in enumerate(self.paths):
                blk = self.blocks[p]
                wp = w64[p][None, :, None]
                xa, eb, gc = xe[:, :, self.x_slices[a]], ee[:, :, self.env_slices[b]], ge[:, :, self.x_slices[cc]]
                # r[e, u, i, j] = sum_k C_ijk g[e, u, k]
                r = (gc.reshape(-1, gc.shape[2]) @ _flat(blk).T).reshape(gc.shape[:2] + blk.shape[:2])
                grad_x[s:t, :, self.x_slices[a]] += wp * np.sum(r * eb[:, :, None, :], axis=3)
                grad_env_edge[s:t, :, self.env_slices[b]] += wp * np.sum(r * xa[:, :, :, None], axis=2)
        grad_env = np.zeros_like(env64)
        np.add.at(grad_env, c, grad_env_edge)
        grad_w, grad_y = env_embed_backward(row_ptr, grad_env, w, Y)
        return grad_x, grad_env, grad_w, grad_y

    def backward_loops(self, row_ptr, x, env, W, g, w, Y):
        x64, env64, w64, g64 = _f64(x), _f64(env), _f64(W), _f64(g)
        wv, yv = _f64(w), _f64(Y)
        c = centers_of_edges(row_ptr)
        n_edges, n_ch, _ = x64.shape
        grad_x = np.zeros_like(x64)
        grad_env = np.zeros_like(env64)
        for e in range(n_edges):
            n = c[e]
            for u in range(n_ch):
                for p, (a, b, cc) in enumerate(self.paths):
                    blk = self.blocks[p]
                    oa, ob, oc = self.x_slices[a].start, self.env_slices[b].start, self.x_slices[cc].start
                    for m1 in range(blk.shape[0]):
                        for m2 in range(blk.shape[1]):
                            for m3 in range(blk.shape[2]):
                                cv = blk[m1, m2, m3]
                                if cv != 0.0:
                                    k = w64[p, u] * cv * g64[e, u, oc + m3]
                                    grad_x[e, u, oa + m1] += k * env64[n, u, ob + m2]
                                    grad_env[n, u, ob + m2] += k * x64[e, u, oa + m1]
        grad_w = np.zeros((n_edges, n_ch))
        grad_y = np.zeros((n_edges, self.d2))
        for e in range(n_edges):
            n = c[e]
            for u in range(n_ch):
                for j in range(self.d2):
                    grad_w[e, u] += grad_env[n, u, j] * yv[e, j]
                    grad_y[e, j] += grad_env[n, u, j] * wv[e, u]
        return grad_x, grad_env, grad_w, grad_y

    # ---- path-weight gradient (training)
    def path_weight_grad(self, row_ptr, x, env, g) -> np.ndarray:
        """grad_W [P, U]: out is linear in W, so this is sum_e <g[e, u, block c], path p's contraction>."""
        x64, env64, g64 = _f64(x), _f64(env), _f64(g)
        c = centers_of_edges(row_ptr)
        n_edges, n_ch, _ = x64.shape
        grad = np.zeros((self.n_paths, n_ch))
        for s in range(0, n_edges, _CHUNK):
            t = min(s + _CHUNK, n_edges)
            xe, ee, ge = x64[s:t], env64[c[s:t]], g64[s:t]
            for (a, b), group in self._groups():
                q = _outer(xe[:, :, self.x_slices[a]], ee[:, :, self.env_slices[b]])
                for p in group:
                    cc = self.paths[p][2]
                    contrib = (q @ _flat(self.blocks[p])).reshape(t - s, n_ch, -1)
                    grad[p] += np.sum(contrib * ge[:, :, self.x_slices[cc]], axis=(0, 2))
        return grad

    def path_weight_grad_loops(self, row_ptr, x, env, g) -> np.ndarray:
        x64, env64, g64 = _f64(x), _f64(env), _f64(g)
        c = centers_of_edges(row_ptr)
        n_edges, n_ch, _ = x64.shape
        grad = np.zeros((self.n_paths, n_ch))
        for e in range(n_edges):
            n = c[e]
            for u in range(n_ch):
                for p, (a, b, cc) in enumerate(self.paths):
                    blk = self.blocks[p]
                    oa, ob, oc = self.x_slices[a].start, self.env_slices[b].start, self.x_slices[cc].start
                    for m1, m2, m3 in zip(*np.nonzero(blk)):
                        grad[p, u] += (blk[m1, m2, m3] * x64[e, u, oa + m1] * env64[n, u, ob + m2]
                                       * g64[e, u, oc + m3])
        return grad
