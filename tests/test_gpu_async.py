"""GPU parity of the bf16 direct-to-LDS GEMM kernels in each of their tile configurations.

The planner picks these kernels only for large bf16 products; here each
configuration (10: 256x256, 11: 256x128, 12: 128x128, 13: 256x256 with 32-deep
k-tiles and a deeper ring, 14 and 15: 256x256 on four waves of 128x128,
64-deep k-tiles in 2 stages or 32-deep in 4; the 256x256 tiles load through
buffer descriptors, the others compute clamped addresses) is
forced through
DLVM_GEMM_CONFIG on shapes that span several tiles and stages with ragged M,
N and K (K a multiple of 8 but not of 64, K smaller than one k-tile), for the
three layouts (forward NN, adjoint wrt the input NT, adjoint wrt the weights
TN), and compared with the oracle.

Inputs are bf16 values, so every product is exact in float32 and a float32
result differs from the float64 oracle only by the summation order: those
comparisons use a bound of 1e-5, tight enough that a lost or doubled k-chunk
fails. bf16 results and derivatives taken from a bf16-rounded saved output use
the bf16 bound.
"""
import re

import numpy as np
import pytest

import oracle
import paper_1711_03016_amd as dl
import workloads
from helpers import TOL, assert_close, device, quant, rel_l2, to_dev, to_np

pytestmark = pytest.mark.gpu

CFGS = [10, 11, 12, 13, 14, 15, 16, 17, 18, 19]
EXACT = 1e-5
ROW_EXACT = 1e-4   # the same, for the worst single row (fewer terms average out)
# (M, N, K): single tile with K = 8, exact tiles, ragged edges with K % 64 != 0,
# many k-tiles (deeper than every ring), and a wide ragged product.
SHAPES = [(8, 136, 8), (256, 256, 64), (520, 264, 200), (1000, 1000, 1000), (264, 520, 2056),
          (1032, 384, 776)]


def _rng(*key):
    return np.random.default_rng(list(key))


@pytest.fixture(params=CFGS)
def cfg(request, monkeypatch):
    monkeypatch.setenv("DLVM_GEMM_CONFIG", str(request.param))
    return request.param


@pytest.mark.parametrize("shape", SHAPES)
def test_async_forward(cfg, shape):
    import torch
    M, N, K = shape
    r = _rng(11, M, N, K)
    X = r.standard_normal((M, K)).astype(np.float32)
    W = (r.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    b = r.uniform(-0.5, 0.5, N).astype(np.float32)
    for act in ("none", "relu", "tanh"):
        for out_dtype in ("f32", "bf16"):
            H = torch.empty((M, N), dtype=torch.float32 if out_dtype == "f32" else torch.bfloat16,
                            device=device())
            dl.dense_forward("bf16", out_dtype, act, M, N, K, 0.75, to_dev(X, "bf16"),
                             to_dev(W, "bf16"), to_dev(b, "bf16"), H)
            torch.cuda.synchronize()
            ref = oracle.dense_forward(quant(X, "bf16"), quant(W, "bf16"), quant(b, "bf16"), act,
                                       0.75)
            if out_dtype == "f32":
                assert_close(to_np(H), ref, EXACT, (act, out_dtype), row_tol=ROW_EXACT)
            else:
                assert_close(to_np(H), ref, TOL["bf16"] / 2, (act, out_dtype), row_tol=TOL["bf16"])


@pytest.mark.parametrize("shape", SHAPES)
def test_async_backward_data(cfg, shape):
    """dX[M,K] = (dY[M,N].W[K,N]^T) * act'(saved output) + R; the contraction runs over N."""
    import torch
    M, N, K = shape
    r = _rng(12, M, N, K)
    u = r.standard_normal((M, K)).astype(np.float32)
    W = (r.standard_normal((K, N)) / np.sqrt(N)).astype(np.float32)
    dY = (r.standard_normal((M, N)) * 0.1).astype(np.float32)
    R = (r.standard_normal((M, K)) * 0.05).astype(np.float32)
    for act in ("none", "relu", "sigmoid"):
        Hprev = oracle.apply_act(quant(u, "f32"), act).astype(np.float32)
        dX = torch.empty((M, K), dtype=torch.float32, device=device())
        dl.dense_backward_data("bf16", "f32", act, M, N, K, to_dev(dY, "bf16"), to_dev(W, "bf16"),
                               to_dev(Hprev, "bf16"), to_dev(R, "f32"), dX)
        torch.cuda.synchronize()
        ref = oracle.dense_vjp_input(quant(u, "f32"), quant(W, "bf16"), quant(dY, "bf16"), act) + R
        # relu' taken from the bf16-rounded output is exact; sigmoid' is not.
        if act != "sigmoid":
            assert_close(to_np(dX), ref, EXACT, act, row_tol=ROW_EXACT)
        else:
            assert_close(to_np(dX), ref, TOL["bf16"], act)


@pytest.mark.parametrize("shape", SHAPES)
def test_async_backward_params(cfg, shape):
    """dW[K,N] = X[M,K]^T.dY[M,N] and db = column sums of dY; the contraction runs over M."""
    import torch
    M, N, K = shape
    r = _rng(13, M, N, K)
    X = r.standard_normal((M, K)).astype(np.float32)
    dY = (r.standard_normal((M, N)) * 0.01).astype(np.float32)
    dW = torch.empty((K, N), dtype=torch.float32, device=device())
    db = torch.empty((N,), dtype=torch.float32, device=device())
    dl.dense_backward_params("bf16", M, N, K, to_dev(X, "bf16"), to_dev(dY, "bf16"), dW, db)
    torch.cuda.synchronize()
    rdW, rdb = oracle.dense_vjp_params(quant(X, "bf16"), quant(dY, "bf16"))
    assert_close(to_np(dW), rdW, EXACT, "dW", row_tol=ROW_EXACT)
    assert_close(to_np(db), rdb, EXACT, "db", row_tol=ROW_EXACT)


def test_async_model_gradient(cfg):
    """The bf16 workload 784-1024-1024-10 at a reduced batch, every product forced onto the
    configuration where it qualifies (its plan names it), against the oracle."""
    import torch
    wl = workloads.WORKLOADS["c3"]
    B = 264
    x, params, y = workloads.make_inputs(wl, B, seed=5)
    m = dl.Model(wl.widths, wl.acts, wl.dtype, wl.loss, False, B)
    names = [e["name"] for e in m.plan(B)]
    assert any(re.search(rf"c{cfg}(s\d+)?$", n) for n in names), names
    dev = device()
    P = m.pack(params, dev, torch.bfloat16)
    ws = torch.empty(m.workspace_bytes(B), dtype=torch.uint8, device=dev)
    loss = torch.empty(1, device=dev)
    dP = torch.full((m.param_count(),), float("nan"), device=dev)
    m.gradient(P, to_dev(x, "bf16"), torch.from_numpy(y.astype(np.int32)).to(dev), B, loss, dP,
               None, ws)
    torch.cuda.synchronize()
    assert m.check(ws) == dl.OK
    spec = oracle.MlpSpec(wl.widths, wl.acts, wl.loss, wl.dtype)
    rl, rg, _ = oracle.mlp_gradient(spec, x, params, y)
    assert abs(loss.item() - rl) <= TOL["bf16"] * abs(rl)
    for l, ((gw, gb), (rw, rb)) in enumerate(zip(m.unpack(dP), rg)):
        assert_close(to_np(gw), rw, TOL["bf16"], ("dW", l))
        assert_close(to_np(gb), rb, TOL["bf16"], ("db", l))
