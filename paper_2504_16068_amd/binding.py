"""ctypes binding of liballegro_tp.so -- argument marshalling only.

Every function here has the name of the C entry point it calls (declared in
include/allegro_tp.h and include/allegro_layer.h), checks tensor shapes, dtypes, devices and contiguity,
allocates outputs with PyTorch when the caller passes none, and hands raw
device pointers plus the current HIP stream to the library.  No arithmetic of
the operation happens in Python, and there is no fallback: if the compiled
library is missing, importing this module raises.
"""

from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liballegro_tp.so")

ALLEGRO_OK = 0
ALLEGRO_E_INVALID = -1
ALLEGRO_E_UNSUPPORTED = -2
ALLEGRO_E_HIP = -3
ALLEGRO_E_NOMEM = -4
ALLEGRO_E_TIMEOUT = -5
ALLEGRO_FULL_PARITY = 1
ALLEGRO_DETERMINISTIC = 2
ALLEGRO_VALIDATE = 4

EXPORTED = (
    "allegro_tp_plan_create", "allegro_tp_plan_destroy", "allegro_tp_plan_query", "allegro_tp_plan_cg",
    "allegro_env_embed", "allegro_tp_forward", "allegro_tp_backward", "allegro_tp_backward_workspace",
    "allegro_tp_backward_train", "allegro_tp_backward_train_noalloc", "allegro_sh_forward", "allegro_sh_backward",
    "allegro_layer_buffers", "allegro_layer_forward", "allegro_layer_backward",
    "allegro_last_error",
)

LAYER_WEIGHTS = ("A", "W", "Mix", "B1", "B2")


class AllegroError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"[{code}] {message}")
        self.code = code


def _load() -> ctypes.CDLL:
    # PyTorch ships its own HIP runtime with the same soname as /opt/rocm's.
    # Loading torch first makes the library bind to that one runtime; loading
    # the library first would put two HIP runtimes in the process.
    import torch  # noqa: F401

    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2504_16068_amd.build.build() or "
                          "__graft_entry__.build() first (there is no CPU fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    ip = ctypes.POINTER(ctypes.c_int)
    lib.allegro_tp_plan_create.argtypes = [ctypes.POINTER(vp), i32, i32, i32]
    lib.allegro_tp_plan_destroy.argtypes = [vp]
    lib.allegro_tp_plan_query.argtypes = [vp, ip, ip, ip, ip, ip]
    lib.allegro_tp_plan_cg.argtypes = [vp, ip, ctypes.POINTER(ctypes.c_double)]
    lib.allegro_env_embed.argtypes = [vp, i64, i64, vp, vp, vp, vp, vp]
    lib.allegro_tp_forward.argtypes = [vp, i64, i64, vp, vp, vp, vp, vp, vp]
    lib.allegro_tp_backward.argtypes = [vp, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.allegro_tp_backward_workspace.argtypes = [vp, i64, ctypes.POINTER(ctypes.c_size_t)]
    lib.allegro_tp_backward_train.argtypes = [vp, i64, i64] + [vp] * 13 + [ctypes.c_size_t, vp]
    lib.allegro_tp_backward_train_noalloc.argtypes = [vp, i64, i64] + [vp] * 13
    lib.allegro_sh_forward.argtypes = [vp, i64, vp, vp, vp]
    lib.allegro_sh_backward.argtypes = [vp, i64, vp, vp, vp, vp]
    szp = ctypes.POINTER(ctypes.c_size_t)
    lib.allegro_layer_buffers.argtypes = [vp, i32, i32, i64, i64, szp, szp]
    lib.allegro_layer_forward.argtypes = [vp, i32, i32, i64, i64] + [vp] * 12 + [ctypes.c_size_t, vp]
    lib.allegro_layer_backward.argtypes = ([vp, i32, i32, i64, i64] + [vp] * 10 + [ctypes.c_size_t] + [vp] * 11
                                           + [ctypes.c_size_t, vp])
    lib.allegro_last_error.restype = ctypes.c_char_p
    for name in EXPORTED:
        if name != "allegro_last_error":
            getattr(lib, name).restype = i32
    return lib


_lib = _load()


def library() -> ctypes.CDLL:
    return _lib


def allegro_last_error() -> str:
    return _lib.allegro_last_error().decode()


def _check(rc: int):
    if rc != ALLEGRO_OK:
        raise AllegroError(rc, allegro_last_error())


class Plan:
    """Owns an allegro_tp_plan*; sizes are read back from the library."""

    def __init__(self, handle: int, lmax: int, U: int, flags: int):
        self.handle = ctypes.c_void_p(handle)
        self.lmax, self.U, self.flags = lmax, U, flags
        d1, d2, np_, nnz = (ctypes.c_int() for _ in range(4))
        _check(_lib.allegro_tp_plan_query(self.handle, ctypes.byref(d1), ctypes.byref(d2), ctypes.byref(np_), None,
                                          ctypes.byref(nnz)))
        self.d1, self.d2, self.n_paths, self.nnz = d1.value, d2.value, np_.value, nnz.value
        # number of x irreps: one per l, or two per l with full parity
        self.n_x = (lmax + 1) * (2 if flags & ALLEGRO_FULL_PARITY else 1)

    def path_desc(self):
        buf = (ctypes.c_int * (6 * self.n_paths))()
        _check(_lib.allegro_tp_plan_query(self.handle, None, None, None, buf, None))
        return [tuple(buf[6 * p:6 * p + 6]) for p in range(self.n_paths)]

    def cg_table(self):
        """(list of (path, i, j, k), list of coefficients) of the sparse combined table."""
        idx = (ctypes.c_int * (4 * self.nnz))()
        val = (ctypes.c_double * self.nnz)()
        _check(_lib.allegro_tp_plan_cg(self.handle, idx, val))
        return [tuple(idx[4 * q:4 * q + 4]) for q in range(self.nnz)], list(val)

    def close(self):
        if self.handle is not None and self.handle.value:
            _lib.allegro_tp_plan_destroy(self.handle)
        self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def allegro_tp_plan_create(lmax: int, U: int, flags: int = ALLEGRO_FULL_PARITY) -> Plan:
    h = ctypes.c_void_p()
    _check(_lib.allegro_tp_plan_create(ctypes.byref(h), int(lmax), int(U), int(flags)))
    return Plan(h.value, lmax, U, flags)


def allegro_tp_plan_destroy(plan: Plan):
    plan.close()


# ----------------------------------------------------------------- tensors

def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None and t.numel() > 0 else ctypes.c_void_p(0)


def _need(t, name, shape, dtype, device):
    import torch

    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device != device or t.device.type != "cuda":
        raise ValueError(f"{name} must live on {device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _stream(stream, device):
    import torch

    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


def _sizes(plan: Plan, row_ptr, n_edges):
    import torch

    if row_ptr.dtype != torch.int64 or row_ptr.dim() != 1 or not row_ptr.is_contiguous():
        raise ValueError("row_ptr must be a contiguous 1-D int64 tensor")
    return row_ptr.numel() - 1, n_edges


def allegro_env_embed(plan: Plan, row_ptr, w, Y, env=None, stream=None):
    import torch

    dev = row_ptr.device
    n, e = _sizes(plan, row_ptr, w.shape[0])
    _need(w, "w", (e, plan.U), torch.float32, dev)
    _need(Y, "Y", (e, plan.d2), torch.float32, dev)
    if env is None:
        env = torch.empty((n, plan.U, plan.d2), device=dev, dtype=torch.float32)
    _need(env, "env", (n, plan.U, plan.d2), torch.float32, dev)
    _check(_lib.allegro_env_embed(plan.handle, n, e, _ptr(row_ptr), _ptr(w), _ptr(Y), _ptr(env),
                                  _stream(stream, dev)))
    return env


def allegro_tp_forward(plan: Plan, row_ptr, x, env, path_w, out=None, stream=None):
    import torch

    dev = row_ptr.device
    n, e = _sizes(plan, row_ptr, x.shape[0])
    _need(x, "x", (e, plan.U, plan.d1), torch.float32, dev)
    _need(env, "env", (n, plan.U, plan.d2), torch.float32, dev)
    _need(path_w, "path_w", (plan.n_paths, plan.U), torch.float32, dev)
    if out is None:
        out = torch.empty_like(x)
    _need(out, "out", (e, plan.U, plan.d1), torch.float32, dev)
    _check(_lib.allegro_tp_forward(plan.handle, n, e, _ptr(row_ptr), _ptr(x), _ptr(env), _ptr(path_w), _ptr(out),
                                   _stream(stream, dev)))
    return out


def allegro_tp_backward(plan: Plan, row_ptr, x, env, path_w, grad_out, w, Y, outs=None, stream=None):
    """Returns (grad_x, grad_env, grad_w, grad_Y)."""
    import torch

    dev = row_ptr.device
    n, e = _sizes(plan, row_ptr, x.shape[0])
    _need(x, "x", (e, plan.U, plan.d1), torch.float32, dev)
    _need(env, "env", (n, plan.U, plan.d2), torch.float32, dev)
    _need(path_w, "path_w", (plan.n_paths, plan.U), torch.float32, dev)
    _need(grad_out, "grad_out", (e, plan.U, plan.d1), torch.float32, dev)
    _need(w, "w", (e, plan.U), torch.float32, dev)
    _need(Y, "Y", (e, plan.d2), torch.float32, dev)
    if outs is None:
        outs = (torch.empty_like(x), torch.empty_like(env), torch.empty_like(w), torch.empty_like(Y))
    gx, genv, gw, gy = outs
    _need(gx, "grad_x", (e, plan.U, plan.d1), torch.float32, dev)
    _need(genv, "grad_env", (n, plan.U, plan.d2), torch.float32, dev)
    _need(gw, "grad_w", (e, plan.U), torch.float32, dev)
    _need(gy, "grad_Y", (e, plan.d2), torch.float32, dev)
    _check(_lib.allegro_tp_backward(plan.handle, n, e, _ptr(row_ptr), _ptr(x), _ptr(env), _ptr(path_w),
                                    _ptr(grad_out), _ptr(w), _ptr(Y), _ptr(gx), _ptr(genv), _ptr(gw), _ptr(gy),
                                    _stream(stream, dev)))
    return gx, genv, gw, gy


def allegro_tp_backward_workspace(plan: Plan, n_centers: int) -> int:
    """Bytes of device workspace allegro_tp_backward_train needs for n_centers."""
    out = ctypes.c_size_t()
    _check(_lib.allegro_tp_backward_workspace(plan.handle, int(n_centers), ctypes.byref(out)))
    return out.value


def allegro_tp_backward_train(plan: Plan, row_ptr, x, env, path_w, grad_out, w, Y, outs=None, workspace=None,
                              stream=None):
    """Returns (grad_x, grad_env, grad_w, grad_Y, grad_path_w); workspace is a uint8 device tensor or None."""
    import torch

    dev = row_ptr.device
    n, e = _sizes(plan, row_ptr, x.shape[0])
    _need(x, "x", (e, plan.U, plan.d1), torch.float32, dev)
    _need(env, "env", (n, plan.U, plan.d2), torch.float32, dev)
    _need(path_w, "path_w", (plan.n_paths, plan.U), torch.float32, dev)
    _need(grad_out, "grad_out", (e, plan.U, plan.d1), torch.float32, dev)
    _need(w, "w", (e, plan.U), torch.float32, dev)
    _need(Y, "Y", (e, plan.d2), torch.float32, dev)
    if outs is None:
        outs = (torch.empty_like(x), torch.empty_like(env), torch.empty_like(w), torch.empty_like(Y),
                torch.empty_like(path_w))
    gx, genv, gw, gy, gpw = outs
    _need(gx, "grad_x", (e, plan.U, plan.d1), torch.float32, dev)
    _need(genv, "grad_env", (n, plan.U, plan.d2), torch.float32, dev)
    _need(gw, "grad_w", (e, plan.U), torch.float32, dev)
    _need(gy, "grad_Y", (e, plan.d2), torch.float32, dev)
    _need(gpw, "grad_path_w", (plan.n_paths, plan.U), torch.float32, dev)
    need = allegro_tp_backward_workspace(plan, n)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    if workspace.device != torch.device(dev) or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous tensor on the same device")
    _check(_lib.allegro_tp_backward_train(plan.handle, n, e, _ptr(row_ptr), _ptr(x), _ptr(env), _ptr(path_w),
                                          _ptr(grad_out), _ptr(w), _ptr(Y), _ptr(gx), _ptr(genv), _ptr(gw),
                                          _ptr(gy), _ptr(gpw), _ptr(workspace),
                                          workspace.numel() * workspace.element_size(), _stream(stream, dev)))
    return gx, genv, gw, gy, gpw


def allegro_tp_backward_train_noalloc(plan: Plan, row_ptr, x, env, path_w, grad_out, w, Y, outs=None, stream=None):
    """Returns (grad_x, grad_env, grad_w, grad_Y, grad_path_w); the library keeps the
    partial sums in its own static device memory (no workspace)."""
    import torch

    dev = row_ptr.device
    n, e = _sizes(plan, row_ptr, x.shape[0])
    _need(x, "x", (e, plan.U, plan.d1), torch.float32, dev)
    _need(env, "env", (n, plan.U, plan.d2), torch.float32, dev)
    _need(path_w, "path_w", (plan.n_paths, plan.U), torch.float32, dev)
    _need(grad_out, "grad_out", (e, plan.U, plan.d1), torch.float32, dev)
    _need(w, "w", (e, plan.U), torch.float32, dev)
    _need(Y, "Y", (e, plan.d2), torch.float32, dev)
    if outs is None:
        outs = (torch.empty_like(x), torch.empty_like(env), torch.empty_like(w), torch.empty_like(Y),
                torch.empty_like(path_w))
    gx, genv, gw, gy, gpw = outs
    _need(gx, "grad_x", (e, plan.U, plan.d1), torch.float32, dev)
    _need(genv, "grad_env", (n, plan.U, plan.d2), torch.float32, dev)
    _need(gw, "grad_w", (e, plan.U), torch.float32, dev)
    _need(gy, "grad_Y", (e, plan.d2), torch.float32, dev)
    _need(gpw, "grad_path_w", (plan.n_paths, plan.U), torch.float32, dev)
    _check(_lib.allegro_tp_backward_train_noalloc(plan.handle, n, e, _ptr(row_ptr), _ptr(x), _ptr(env), _ptr(path_w),
                                                  _ptr(grad_out), _ptr(w), _ptr(Y), _ptr(gx), _ptr(genv), _ptr(gw),
                                                  _ptr(gy), _ptr(gpw), _stream(stream, dev)))
    return gx, genv, gw, gy, gpw


def allegro_sh_forward(plan: Plan, vec, Y=None, stream=None):
    """Y [E, d2] float32 from edge vectors vec [E, 3] float64."""
    import torch

    dev = vec.device
    e = vec.shape[0]
    _need(vec, "vec", (e, 3), torch.float64, dev)
    if Y is None:
        Y = torch.empty((e, plan.d2), device=dev, dtype=torch.float32)
    _need(Y, "Y", (e, plan.d2), torch.float32, dev)
    _check(_lib.allegro_sh_forward(plan.handle, e, _ptr(vec), _ptr(Y), _stream(stream, dev)))
    return Y


def allegro_sh_backward(plan: Plan, vec, grad_Y, grad_vec=None, stream=None):
    """grad_vec [E, 3] float64 from vec [E, 3] float64 and grad_Y [E, d2] float32."""
    import torch

    dev = vec.device
    e = vec.shape[0]
    _need(vec, "vec", (e, 3), torch.float64, dev)
    _need(grad_Y, "grad_Y", (e, plan.d2), torch.float32, dev)
    if grad_vec is None:
        grad_vec = torch.empty((e, 3), device=dev, dtype=torch.float64)
    _need(grad_vec, "grad_vec", (e, 3), torch.float64, dev)
    _check(_lib.allegro_sh_backward(plan.handle, e, _ptr(vec), _ptr(grad_Y), _ptr(grad_vec), _stream(stream, dev)))
    return grad_vec


# ------------------------------------------------------------------- layer

def layer_weight_shapes(plan: Plan, L: int, H: int):
    """Shapes of the weights of one layer (include/allegro_layer.h)."""
    return {"A": (L, plan.U), "W": (plan.n_paths, plan.U), "Mix": (plan.n_x, plan.U, plan.U),
            "B1": (L + plan.U, H), "B2": (H, L)}


def allegro_layer_buffers(plan: Plan, L: int, H: int, n_centers: int, n_edges: int):
    """(saved_bytes, workspace_bytes) of one layer."""
    sv, ws = ctypes.c_size_t(), ctypes.c_size_t()
    _check(_lib.allegro_layer_buffers(plan.handle, int(L), int(H), int(n_centers), int(n_edges), ctypes.byref(sv),
                                      ctypes.byref(ws)))
    return sv.value, ws.value


def _bytes_buffer(t, need, name, device):
    import torch

    if t is None:
        return torch.empty(max(need, 16), dtype=torch.uint8, device=device)
    if t.device != torch.device(device) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous tensor on {device}")
    return t


def _nbytes(t):
    return t.numel() * t.element_size()


def _layer_inputs(plan, L, H, row_ptr, h, V, Y, weights):
    import torch

    dev = row_ptr.device
    n, e = _sizes(plan, row_ptr, V.shape[0])
    _need(h, "h", (e, L), torch.float32, dev)
    _need(V, "V", (e, plan.U, plan.d1), torch.float32, dev)
    _need(Y, "Y", (e, plan.d2), torch.float32, dev)
    for name, shape in layer_weight_shapes(plan, L, H).items():
        _need(weights[name], name, shape, torch.float32, dev)
    return dev, n, e


def allegro_layer_forward(plan: Plan, L: int, H: int, row_ptr, h, V, Y, weights, h_out=None, V_out=None,
                          saved=None, stream=None):
    """Returns (h_out, V_out, saved); weights maps A, W, Mix, B1, B2 to device tensors."""
    import torch

    dev, n, e = _layer_inputs(plan, L, H, row_ptr, h, V, Y, weights)
    sv_need, _ = allegro_layer_buffers(plan, L, H, n, e)
    h_out = torch.empty_like(h) if h_out is None else h_out
    V_out = torch.empty_like(V) if V_out is None else V_out
    _need(h_out, "h_out", (e, L), torch.float32, dev)
    _need(V_out, "V_out", (e, plan.U, plan.d1), torch.float32, dev)
    saved = _bytes_buffer(saved, sv_need, "saved", dev)
    _check(_lib.allegro_layer_forward(plan.handle, int(L), int(H), n, e, _ptr(row_ptr), _ptr(h), _ptr(V), _ptr(Y),
                                      *(_ptr(weights[k]) for k in LAYER_WEIGHTS), _ptr(h_out), _ptr(V_out),
                                      _ptr(saved), _nbytes(saved), _stream(stream, dev)))
    return h_out, V_out, saved


def allegro_layer_backward(plan: Plan, L: int, H: int, row_ptr, h, V, Y, weights, saved, dh_out, dV_out,
                           outs=None, workspace=None, stream=None):
    """Returns a dict of gradients: h, V, Y and the weights A, W, Mix, B1, B2."""
    import torch

    dev, n, e = _layer_inputs(plan, L, H, row_ptr, h, V, Y, weights)
    _need(dh_out, "dh_out", (e, L), torch.float32, dev)
    _need(dV_out, "dV_out", (e, plan.U, plan.d1), torch.float32, dev)
    _, ws_need = allegro_layer_buffers(plan, L, H, n, e)
    if outs is None:
        outs = {"h": torch.empty_like(h), "V": torch.empty_like(V), "Y": torch.empty_like(Y)}
        outs.update({k: torch.empty_like(weights[k]) for k in LAYER_WEIGHTS})
    _need(outs["h"], "dh", (e, L), torch.float32, dev)
    _need(outs["V"], "dV", (e, plan.U, plan.d1), torch.float32, dev)
    _need(outs["Y"], "dY", (e, plan.d2), torch.float32, dev)
    for name, shape in layer_weight_shapes(plan, L, H).items():
        _need(outs[name], "d" + name, shape, torch.float32, dev)
    workspace = _bytes_buffer(workspace, ws_need, "workspace", dev)
    _check(_lib.allegro_layer_backward(plan.handle, int(L), int(H), n, e, _ptr(row_ptr), _ptr(h), _ptr(V), _ptr(Y),
                                       *(_ptr(weights[k]) for k in LAYER_WEIGHTS), _ptr(saved), _nbytes(saved),
                                       _ptr(dh_out), _ptr(dV_out), _ptr(outs["h"]), _ptr(outs["V"]), _ptr(outs["Y"]),
                                       *(_ptr(outs[k]) for k in LAYER_WEIGHTS), _ptr(workspace), _nbytes(workspace),
                                       _stream(stream, dev)))
    return outs
