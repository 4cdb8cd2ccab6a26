"""The allocation-free training backward (static device scratch) against the
training backward with a caller workspace, through the C ABI.

Two calls in a row on one plan, the second with a smaller input, so the
second call finds the first call's partial sums in the shared scratch.  At
lmax < 3 the first input has more centers than one chunk of the scratch holds,
so the chunk loop and the final sum over chunk rows are exercised; grad_path_w
is then the same sum in another fixed order and must agree to the backward
tolerance.  At lmax 3 the matrix-core kernel's per-wave rows fit the scratch
at any size: one launch and the same reduction as the workspace version, so
grad_path_w must be bit-identical too.  grad_x, grad_env, grad_w and grad_Y
come from the same kernels as the workspace version and must be bit-identical.
"""

import sys

import numpy as np
import pytest

import workloads
from tests.parity import BWD_TOL, block_rel_err

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
DEV = "cuda:0"


def _note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _inputs(plan, degrees, seed):
    g = torch.Generator(device=DEV).manual_seed(seed)
    rp = torch.from_numpy(np.concatenate([[0], np.cumsum(degrees)]).astype(np.int64)).to(DEV)
    n, e = len(degrees), int(np.sum(degrees))
    x = torch.randn((e, plan.U, plan.d1), generator=g, device=DEV)
    gr = torch.randn((e, plan.U, plan.d1), generator=g, device=DEV)
    w = torch.randn((e, plan.U), generator=g, device=DEV)
    y = torch.randn((e, plan.d2), generator=g, device=DEV)
    pw = torch.randn((plan.n_paths, plan.U), generator=g, device=DEV) / np.sqrt(plan.n_paths)
    env = torch.randn((n, plan.U, plan.d2), generator=g, device=DEV)
    return rp, x, env, pw, gr, w, y


@pytest.mark.parametrize("lmax,U", [(3, 128), (2, 64)])
def test_noalloc_matches_workspace_version(lmax, U):
    import paper_2504_16068_amd as at

    plan = at.allegro_tp_plan_create(lmax, U, at.ALLEGRO_FULL_PARITY)
    cols = plan.n_paths * U
    chunk = (16 << 20) // cols - 128 - 256
    rng = np.random.default_rng(lmax * 1000 + U)
    # first call: a bit over two chunks of centers (with empty segments); second: fewer centers
    sizes = (2 * chunk + 77, chunk // 3)
    for call, n in enumerate(sizes):
        degrees = rng.poisson(6.0, n)
        degrees[rng.integers(0, n, n // 50)] = 0
        _note(f"[gpu] no-alloc training backward lmax={lmax} U={U} call {call}: N={n} E={int(degrees.sum())}")
        rp, x, env, pw, gr, w, y = _inputs(plan, degrees, seed=17 + call)
        ws = torch.empty(at.allegro_tp_backward_workspace(plan, n), dtype=torch.uint8, device=DEV)
        ref = at.allegro_tp_backward_train(plan, rp, x, env, pw, gr, w, y, workspace=ws)
        got = at.allegro_tp_backward_train_noalloc(plan, rp, x, env, pw, gr, w, y)
        torch.cuda.synchronize()
        for name, a, b in zip(("grad_x", "grad_env", "grad_w", "grad_Y"), got[:4], ref[:4]):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), name
        if lmax >= 3:
            assert torch.equal(got[4].view(torch.int32), ref[4].view(torch.int32)), "grad_path_w"
            del ws, ref, got
            continue
        err = block_rel_err(got[4].cpu().numpy(), ref[4].cpu().numpy())
        _note(f"  grad_path_w err vs workspace version {err:.2e}")
        assert err <= BWD_TOL
        # fp64 sum of the per-center rows ([P][U]) the workspace version wrote
        rows = ws[: n * cols * 4].view(torch.float32)
        part = np.ascontiguousarray(rows.cpu().numpy()).reshape(n, cols).astype(np.float64)
        total = part.sum(axis=0)
        got_pw = got[4].cpu().numpy().reshape(cols).astype(np.float64)
        # recursive-summation bound: per chunk ceil(ceil(rows / 128) / 4) + 2 additions in a
        # range, 128 over the ranges, then at most 256 over the chunk rows
        depth = -(-(-(-chunk // 128)) // 4) + 2 + 128 + 256
        bound = 1.01 * depth * 2.0 ** -24 * np.abs(part).sum(axis=0)
        assert np.all(np.abs(got_pw - total) <= bound)
        del ws, ref, got
