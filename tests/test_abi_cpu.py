"""Host-side tests of the C ABI (no GPU): exports, plans, coupling table, errors.

The coupling table of the library comes from its own C++ builder (null space of
the so(3) intertwiner equations); here it is compared, as outputs only, with
the oracle's table (Racah's formula plus the change of basis).  Error paths are
exercised only where the library rejects the call before any HIP call.
"""

import ctypes
import os
import re

import numpy as np
import pytest

from oracle import cg as ocg
from oracle import irreps as oirreps

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("allegro_tp.h", "allegro_layer.h")]

binding = pytest.importorskip("paper_2504_16068_amd.binding",
                              reason="liballegro_tp.so not built (run __graft_entry__.build())")


def _declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(allegro_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = binding.library()
    names = _declared_functions()
    assert set(names) == set(binding.EXPORTED)
    for name in names:
        assert hasattr(lib, name), name


def _declared_arities():
    """Number of parameters of every function the headers declare."""
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    out = {}
    for name, params in re.findall(r"\b(allegro_\w+)\s*\(([^;{]*?)\)\s*;", text, flags=re.S):
        params = params.strip()
        out[name] = 0 if params in ("", "void") else params.count(",") + 1
    return out


def test_binding_argument_counts_match_headers():
    lib = binding.library()
    arities = _declared_arities()
    assert set(arities) == set(binding.EXPORTED)
    for name, n in arities.items():
        fn = getattr(lib, name)
        if fn.argtypes is not None:
            assert len(fn.argtypes) == n, (name, len(fn.argtypes), n)


def test_layer_rejects_bad_arguments_before_any_launch():
    lib = binding.library()
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    ok_ptr, ok_rp, bad_ptr = vp(0x10000), vp(0x20000), vp(0x10004)
    plan = binding.allegro_tp_plan_create(2, 64, binding.ALLEGRO_FULL_PARITY)
    sv, ws = binding.allegro_layer_buffers(plan, 64, 128, 10, 100)
    d1, d2, P, U, L, H = plan.d1, plan.d2, plan.n_paths, 64, 64, 128
    f = 4
    # saved: w, env, T, s, a; each region rounded up to 256 bytes
    up = lambda b: (b + 255) // 256 * 256  # noqa: E731
    assert sv == up(100 * U * f) + up(10 * U * d2 * f) + up(100 * U * d1 * f) + up(100 * U * f) + up(100 * H * f)
    assert ws > up(100 * U * d1 * f) + binding.allegro_tp_backward_workspace(plan, 10)
    with pytest.raises(binding.AllegroError) as ex:
        binding.allegro_layer_buffers(plan, 48, 128, 10, 100)
    assert ex.value.code == binding.ALLEGRO_E_UNSUPPORTED and "L=48" in str(ex.value)
    plan32 = binding.allegro_tp_plan_create(2, 32, binding.ALLEGRO_FULL_PARITY)
    with pytest.raises(binding.AllegroError) as ex:
        binding.allegro_layer_buffers(plan32, 64, 64, 10, 100)
    assert ex.value.code == binding.ALLEGRO_E_UNSUPPORTED and "U=64" in str(ex.value)
    plan32.close()
    fwd = [plan.handle, L, H, 10, 100, ok_rp] + [ok_ptr] * 10
    rc, msg = _err(lib.allegro_layer_forward, *fwd, ok_ptr, sz(sv - 1), None)
    assert rc == binding.ALLEGRO_E_INVALID and "saved" in msg
    rc, msg = _err(lib.allegro_layer_forward, *fwd, bad_ptr, sz(sv), None)
    assert rc == binding.ALLEGRO_E_INVALID and "saved" in msg and "aligned" in msg
    bad = list(fwd)
    bad[8] = None  # Y
    rc, msg = _err(lib.allegro_layer_forward, *bad, ok_ptr, sz(sv), None)
    assert rc == binding.ALLEGRO_E_INVALID and "Y is NULL" in msg
    rc, msg = _err(lib.allegro_layer_forward, plan.handle, L, H, 0, 5, *([ok_ptr] * 12), sz(sv), None)
    assert rc == binding.ALLEGRO_E_INVALID and "N=0" in msg
    bwd = [plan.handle, L, H, 10, 100] + [ok_ptr] * 10
    rc, msg = _err(lib.allegro_layer_backward, *bwd, sz(sv), *([ok_ptr] * 11), sz(ws - 1), None)
    assert rc == binding.ALLEGRO_E_INVALID and "workspace" in msg
    grads = [ok_ptr] * 11
    grads[5] = None  # dA
    rc, msg = _err(lib.allegro_layer_backward, *bwd, sz(sv), *grads, sz(ws), None)
    assert rc == binding.ALLEGRO_E_INVALID and "dA is NULL" in msg
    plan.close()


CONFIGS = [(lmax, full, u) for lmax in (1, 2, 3) for full in (False, True) for u in (16, 32, 64, 128)]


@pytest.mark.parametrize("lmax,full,U", CONFIGS)
def test_plan_sizes_and_paths_match_oracle(lmax, full, U):
    flags = binding.ALLEGRO_FULL_PARITY if full else 0
    plan = binding.allegro_tp_plan_create(lmax, U, flags)
    xs, es = oirreps.x_irreps(lmax, full), oirreps.env_irreps(lmax)
    assert plan.d1 == oirreps.dim(xs) and plan.d2 == oirreps.dim(es)
    ps = oirreps.paths(lmax, full)
    assert plan.n_paths == len(ps)
    expect = [(xs[a][0], xs[a][1], es[b][0], es[b][1], xs[c][0], xs[c][1]) for a, b, c in ps]
    assert plan.path_desc() == expect
    plan.close()


@pytest.mark.parametrize("lmax,full", [(1, False), (1, True), (2, False), (2, True), (3, False), (3, True)])
def test_coupling_table_matches_oracle(lmax, full):
    plan = binding.allegro_tp_plan_create(lmax, 64, binding.ALLEGRO_FULL_PARITY if full else 0)
    idx, val = plan.cg_table()
    ref = ocg.combined_sparse(lmax, full)
    assert plan.nnz == len(ref) == len(idx)
    got = {k: v for k, v in zip(idx, val)}
    want = {(p, i, j, k): v for p, i, j, k, v in ref}
    assert set(got) == set(want)
    err = max(abs(got[k] - want[k]) for k in want)
    assert err <= 1e-14, err


def _err(fn, *args):
    rc = fn(*args)
    return rc, binding.allegro_last_error()


def test_plan_create_rejects_bad_arguments():
    lib = binding.library()
    h = ctypes.c_void_p()
    rc, msg = _err(lib.allegro_tp_plan_create, ctypes.byref(h), 4, 64, 1)
    assert rc == binding.ALLEGRO_E_UNSUPPORTED and "lmax" in msg and not h.value
    rc, msg = _err(lib.allegro_tp_plan_create, ctypes.byref(h), 2, 48, 1)
    assert rc == binding.ALLEGRO_E_UNSUPPORTED and "U=48" in msg
    rc, msg = _err(lib.allegro_tp_plan_create, ctypes.byref(h), 2, 64, 64)
    assert rc == binding.ALLEGRO_E_INVALID and "flags" in msg
    rc, _ = _err(lib.allegro_tp_plan_create, None, 2, 64, 1)
    assert rc == binding.ALLEGRO_E_INVALID
    with pytest.raises(binding.AllegroError) as ex:
        binding.allegro_tp_plan_create(0, 64)
    assert ex.value.code == binding.ALLEGRO_E_UNSUPPORTED
    assert lib.allegro_tp_plan_destroy(None) == binding.ALLEGRO_OK


@pytest.mark.parametrize("where,flags", [("plan", 1), ("table", 1), ("status", 1 | 4)])
def test_plan_create_reports_allocation_failure(monkeypatch, where, flags):
    """A simulated out-of-memory in each allocation of plan creation returns
    ALLEGRO_E_NOMEM, leaves *plan NULL and names the allocation; the status
    word (ALLEGRO_VALIDATE) fails before any HIP call."""
    lib = binding.library()
    h = ctypes.c_void_p(0x1234)
    monkeypatch.setenv("ALLEGRO_SIMULATE_ALLOC_FAILURE", where)
    rc, msg = _err(lib.allegro_tp_plan_create, ctypes.byref(h), 3, 128, flags)
    assert rc == binding.ALLEGRO_E_NOMEM and not h.value
    assert {"plan": "plan allocation", "table": "table allocation", "status": "status word"}[where] in msg
    with pytest.raises(binding.AllegroError) as ex:
        binding.allegro_tp_plan_create(3, 128, flags)
    assert ex.value.code == binding.ALLEGRO_E_NOMEM
    monkeypatch.delenv("ALLEGRO_SIMULATE_ALLOC_FAILURE")
    if where != "status":  # without the hook the same call succeeds (no GPU needed)
        rc, _ = _err(lib.allegro_tp_plan_create, ctypes.byref(h), 3, 128, flags)
        assert rc == binding.ALLEGRO_OK and h.value
        assert lib.allegro_tp_plan_destroy(h) == binding.ALLEGRO_OK


def test_entry_points_reject_bad_arguments_before_any_launch():
    lib = binding.library()
    plan = binding.allegro_tp_plan_create(2, 64, binding.ALLEGRO_FULL_PARITY)
    h = plan.handle
    vp = ctypes.c_void_p
    ok_ptr, ok_rp, bad_ptr = vp(0x10000), vp(0x20000), vp(0x10004)
    # null plan
    rc, msg = _err(lib.allegro_env_embed, None, 1, 1, ok_rp, ok_ptr, ok_ptr, ok_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "plan" in msg
    # negative sizes, edges without centers, huge N
    rc, msg = _err(lib.allegro_tp_forward, h, -1, 5, ok_rp, ok_ptr, ok_ptr, ok_ptr, ok_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "negative" in msg
    rc, msg = _err(lib.allegro_tp_forward, h, 0, 5, ok_rp, ok_ptr, ok_ptr, ok_ptr, ok_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "N=0" in msg
    rc, msg = _err(lib.allegro_tp_forward, h, 1 << 31, 5, ok_rp, ok_ptr, ok_ptr, ok_ptr, ok_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "2^31" in msg
    # null / misaligned tensors
    rc, msg = _err(lib.allegro_tp_forward, h, 3, 5, ok_rp, None, ok_ptr, ok_ptr, ok_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "x is NULL" in msg
    rc, msg = _err(lib.allegro_tp_forward, h, 3, 5, ok_rp, bad_ptr, ok_ptr, ok_ptr, ok_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "aligned" in msg
    rc, msg = _err(lib.allegro_tp_forward, h, 3, 5, vp(0x20004), ok_ptr, ok_ptr, ok_ptr, ok_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "row_ptr" in msg
    rc, msg = _err(lib.allegro_tp_backward, h, 3, 5, ok_rp, ok_ptr, ok_ptr, ok_ptr, ok_ptr, ok_ptr, ok_ptr,
                   ok_ptr, ok_ptr, ok_ptr, bad_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "grad_Y" in msg
    rc, msg = _err(lib.allegro_env_embed, h, 3, 5, ok_rp, ok_ptr, None, ok_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "Y is NULL" in msg
    rc, msg = _err(lib.allegro_sh_forward, h, 4, bad_ptr, ok_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "vec" in msg
    rc, msg = _err(lib.allegro_sh_backward, h, -1, ok_ptr, ok_ptr, ok_ptr, None)
    assert rc == binding.ALLEGRO_E_INVALID and "negative" in msg
    rc, msg = _err(lib.allegro_sh_backward, h, 4, ok_ptr, ok_ptr, None, None)
    assert rc == binding.ALLEGRO_E_INVALID and "grad_vec is NULL" in msg
    assert lib.allegro_sh_forward(h, 0, None, None, None) == binding.ALLEGRO_OK
    # training backward: workspace size is host arithmetic; missing / short workspace is rejected
    assert binding.allegro_tp_backward_workspace(plan, 10) == (10 + 128) * plan.n_paths * 64 * 4
    args = [h, 3, 5, ok_rp] + [ok_ptr] * 11
    rc, msg = _err(lib.allegro_tp_backward_train, *args, None, 1 << 20, None)
    assert rc == binding.ALLEGRO_E_INVALID and "workspace is NULL" in msg
    rc, msg = _err(lib.allegro_tp_backward_train, *args, ok_ptr, 100, None)
    assert rc == binding.ALLEGRO_E_INVALID and "smaller" in msg
    args[14] = None
    rc, msg = _err(lib.allegro_tp_backward_train, *args, ok_ptr, 1 << 20, None)
    assert rc == binding.ALLEGRO_E_INVALID and "grad_path_w is NULL" in msg
    # empty problem: successful no-op
    for fn, nargs in ((lib.allegro_env_embed, 5), (lib.allegro_tp_forward, 6), (lib.allegro_tp_backward, 12)):
        rc = fn(h, 0, 0, *([None] * (nargs - 1)), None)
        assert rc == binding.ALLEGRO_OK
    plan.close()


def test_noalloc_rejects_too_many_centers_before_any_launch():
    lib = binding.library()
    vp = ctypes.c_void_p
    ok_ptr, ok_rp = vp(0x10000), vp(0x20000)
    # per-center rows (lmax < 3; the matrix-core kernel's per-wave rows at lmax 3 have no such limit)
    plan = binding.allegro_tp_plan_create(2, 128, binding.ALLEGRO_FULL_PARITY)
    cols = plan.n_paths * 128
    chunk = (16 << 20) // cols - 128 - 256
    assert chunk == 3985
    n = 256 * chunk + 1
    rc = lib.allegro_tp_backward_train_noalloc(plan.handle, n, 10, ok_rp, *([ok_ptr] * 12), None)
    assert rc == binding.ALLEGRO_E_INVALID
    assert "allocation-free maximum" in binding.allegro_last_error()
    plan.close()
