"""GPU parity of matrix multiplication reordering (§3.1.2): the chain product
run in the library's optimal order, and in caller-given orders, against the
oracle's left-to-right float64 product; the order itself against the
oracle's recurrence."""
import numpy as np
import pytest

import oracle
import paper_1711_03016_amd as dl
import workloads
from helpers import TOL, device, rel_l2, to_dev, to_np

pytestmark = pytest.mark.gpu


def _left_to_right(n):
    return [[(j - 1 if j > i else -1) for j in range(n)] for i in range(n)]


def _run(dtype, dims, mats, split=None):
    import torch
    dev = device()
    dm = [to_dev(m, dtype) for m in mats]
    out = torch.full((dims[0], dims[-1]), float("nan"), device=dev)
    nb = dl.matrix_chain_ws_bytes(dtype, dims, split)
    ws = torch.empty(max(nb, 16), dtype=torch.uint8, device=dev)
    dl.matrix_chain(dtype, dims, dm, out, ws, split)
    torch.cuda.synchronize()
    return to_np(out)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seed", range(6))
def test_random_chains(dtype, seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(2, 7))
    dims = [int(v) for v in rng.integers(1, 300, size=n + 1)]
    if seed % 2 == 0:                       # 16-byte rows: the direct-to-LDS kernels
        dims = [8 * ((v + 7) // 8) for v in dims]
    mats = workloads.make_chain_inputs(dims, seed=seed)
    ref = oracle.chain_product(mats, dtype)
    tol = TOL[dtype]
    assert rel_l2(_run(dtype, dims, mats), ref) <= tol
    assert rel_l2(_run(dtype, dims, mats, _left_to_right(n)), ref) <= tol


def test_textbook_chain_every_order_gives_the_product():
    dims = [30, 35, 15, 5, 10, 20, 25]
    mats = workloads.make_chain_inputs(dims, seed=4)
    ref = oracle.chain_product(mats)
    cost, split = dl.chain_order(dims)
    assert (cost, split) == oracle.chain_order(dims)
    for sp in (split, _left_to_right(6), None):
        assert rel_l2(_run("f32", dims, mats, sp), ref) <= 1e-5


def test_m1_full_size():
    """The m1 chain at its full size, optimal and left-to-right orders."""
    wl = workloads.CHAIN_WORKLOADS["m1"]
    mats = workloads.make_chain_inputs(wl.dims)
    ref = oracle.chain_product(mats, wl.dtype)
    assert rel_l2(_run(wl.dtype, wl.dims, mats), ref) <= TOL[wl.dtype]
    assert rel_l2(_run(wl.dtype, wl.dims, mats, _left_to_right(wl.n)), ref) <= TOL[wl.dtype]
    cost, _ = dl.chain_order(wl.dims)
    d = wl.dims
    l2r = sum(d[0] * d[k + 1] * d[k + 2] for k in range(wl.n - 1))
    assert cost < l2r / 2


def test_chain_handle_matches_stateless_call():
    """dlvm_chain_run (a handle with the order fixed) computes bit for bit what
    dlvm_matrix_chain computes for the same order."""
    import torch
    wl = workloads.CHAIN_WORKLOADS["m1"]
    dims = list(wl.dims)
    mats = workloads.make_chain_inputs(dims, seed=8)
    dev = device()
    dm = [to_dev(m, wl.dtype) for m in mats]
    h = dl.Chain(wl.dtype, dims)
    ws = torch.empty(h.workspace_bytes(1), dtype=torch.uint8, device=dev)
    a = torch.empty((dims[0], dims[-1]), device=dev)
    h.run(dm, a, ws)
    b = torch.empty_like(a)
    dl.matrix_chain(wl.dtype, dims, dm, b, ws)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert sum(p["flops"] for p in h.plan(1)) == 2 * dl.chain_order(dims)[0]


@pytest.mark.parametrize("dims", [
    [1, 1, 1],                         # two 1 x 1 matrices
    [1, 300, 1],                       # a dot product
    [300, 1, 300],                     # an outer product
    [17, 1, 9, 1, 33],
])
def test_degenerate_chains(dims):
    mats = workloads.make_chain_inputs(dims, seed=12)
    ref = oracle.chain_product(mats)
    assert rel_l2(_run("f32", dims, mats), ref) <= 1e-5
    assert rel_l2(_run("bf16", dims, mats), oracle.chain_product(mats, "bf16")) <= TOL["bf16"]


def test_longest_chain():
    """32 matrices (the maximum), shapes 1..24."""
    rng = np.random.default_rng(77)
    dims = [int(v) for v in rng.integers(1, 25, size=33)]
    mats = workloads.make_chain_inputs(dims, seed=13)
    ref = oracle.chain_product(mats)
    cost, split = dl.chain_order(dims)
    assert (cost, split) == oracle.chain_order(dims)
    assert rel_l2(_run("f32", dims, mats), ref) <= 1e-5
