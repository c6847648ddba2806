"""The allocation-free forward (sinkhorn_forward_noalloc, scratch in the
library's fixed per-GPU array) against sinkhorn_forward (scratch in a caller
workspace) through the C ABI: two calls in a row, the second with a smaller
input, each bit-identical to the workspace entry point and within the parity
tolerances of the fp64 oracle.  Problems too large for the array are refused
before anything is launched."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_1907_01729_amd as sk
import workloads
from parity_util import LOSS_RTOL, POT_ATOL, gauge_fixed_errors, loss_rel_err

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _run_both(prob):
    mu, nu, C = _t(prob.mu), _t(prob.nu), _t(prob.C)
    ref = sk.sinkhorn_forward(mu, nu, C, prob.lam, prob.n_iter, prob.tol)
    out = sk.sinkhorn_forward_noalloc(mu, nu, C, prob.lam, prob.n_iter, prob.tol)
    torch.cuda.synchronize()
    return ({k: v.cpu().numpy() for k, v in out.items()}, {k: v.cpu().numpy() for k, v in ref.items()})


def _check(prob):
    need = sk.sinkhorn_workspace_bytes(prob.B, prob.d1, prob.d2, int(prob.c_batched), prob.lam, prob.n_iter,
                                       prob.tol)
    print(f"[noalloc] {prob.name} B={prob.B} d1={prob.d1} d2={prob.d2} workspace={need}", file=sys.stderr,
          flush=True)
    assert need <= sk.NOALLOC_SCRATCH_BYTES
    got, ref = _run_both(prob)
    for k in ref:
        np.testing.assert_array_equal(got[k], ref[k], err_msg=k)
    o = oracle.forward(prob.mu, prob.nu, prob.C, prob.lam, prob.n_iter, n_iter_b=got["iters"])
    assert loss_rel_err(got["loss"], o["loss"]) <= LOSS_RTOL
    ea, eb = gauge_fixed_errors(prob.mu, prob.nu, got["alpha"], got["beta"], o["alpha"], o["beta"])
    assert ea <= POT_ATOL and eb <= POT_ATOL


def test_noalloc_matches_workspace_forward_two_calls():
    """A shared-cost tiled problem (image histograms, 16 per batch), then a
    smaller per-sample-cost tiled problem on the same scratch: stale contents
    of the first call must not reach the second."""
    first = workloads.make_config(3, B=16, n_iter=40)
    second = workloads.random_problem(seed=901, B=3, d1=150, d2=260, lam=0.08, n_iter=30, c_batched=True,
                                      zero_frac=0.1)
    assert sk.sinkhorn_workspace_bytes(second.B, second.d1, second.d2, 1, second.lam, 30) < \
        sk.sinkhorn_workspace_bytes(first.B, first.d1, first.d2, 0, first.lam, 40)
    _check(first)
    _check(second)


def test_noalloc_early_stop_and_resident():
    """An early-stopped shared-cost batch (the stop test's counters live in the
    scratch), then a resident problem that needs no scratch at all."""
    first = workloads.random_problem(seed=902, B=10, d1=180, d2=200, lam=0.1, n_iter=300, tol=2e-4)
    second = workloads.random_problem(seed=903, B=5, d1=40, d2=30, lam=0.1, n_iter=50)
    _check(first)
    _check(second)


def test_noalloc_split_merge_twice():
    """Rows wider than 1024 columns with an early stop, twice in a row on the
    same scratch: the merge's per-problem stop accumulators left by the first
    call are cleared before the second uses them."""
    prob = workloads.random_problem(seed=904, B=6, d1=150, d2=2100, lam=0.05, n_iter=120, tol=1e-3,
                                    cost="grid1d")
    _check(prob)
    _check(prob)


def test_noalloc_rejects_problems_beyond_the_scratch():
    """The grid workload's workspace exceeds the fixed array: refused with
    SK_ERR_WORKSPACE before any launch (no allocation, no partial result)."""
    B, d = 64, 4096
    need = sk.sinkhorn_workspace_bytes(B, d, d, 0, 1e-3, 500, 1e-6)
    assert need > sk.NOALLOC_SCRATCH_BYTES
    mu = torch.full((B, d), 1.0 / d, device=DEV)
    C = torch.zeros((d, d), device=DEV)
    with pytest.raises(sk.SinkhornError) as e:
        sk.sinkhorn_forward_noalloc(mu, mu, C, 1e-3, 500, 1e-6)
    assert e.value.status == -5
