"""GPU parity of the recurrent cell (§3.1.2's linear-algebra fusion of
h_t = f(W x_{t-1} + U h_{t-1} + b)) against the oracle's unfused RNN.

The product computes each step as one product over the concatenated
contraction [xs[t] hs[t]] . [W; U]; the oracle as two products and two
additions. Shapes cover ragged batch rows, contraction phases that end inside
a k-tile, operands whose rows rule out 16-byte loads, every tile
configuration, and the full r1 workload (at a reduced batch, and at its full
batch with repeated rows).
"""
from dataclasses import replace

import numpy as np
import pytest

import oracle
import paper_1711_03016_amd as dl
import workloads
from helpers import TOL, device, rel_l2, to_dev, to_np, torch_dtype

pytestmark = pytest.mark.gpu


def _case(T, Kx, H, B, dtype, act, seed=None):
    wl = replace(workloads.RNN_WORKLOADS["r1"], steps=T, in_width=Kx, hidden=H, dtype=dtype,
                 act=act, batch=B)
    return wl, workloads.make_rnn_inputs(wl, seed=seed)


def _spec(wl):
    return oracle.RnnSpec(wl.steps, wl.in_width, wl.hidden, wl.act, wl.dtype)


@pytest.mark.parametrize("dtype,act,M,Kx,H", [
    ("f32", "tanh", 37, 40, 72),       # 16-byte rows, phases end inside a k-tile
    ("f32", "relu", 64, 37, 33),       # odd widths: element-wise loads
    ("bf16", "tanh", 300, 96, 128),    # direct-to-LDS kernels
    ("bf16", "sigmoid", 45, 36, 20),   # Kx % 8 != 0: register-staged kernel
    ("bf16", "none", 256, 1024, 1024),
])
def test_cell_forward(dtype, act, M, Kx, H):
    wl, (xs, h0, W, U, b, _) = _case(1, Kx, H, M, dtype, act)
    dev = device()
    WU = to_dev(np.concatenate([W, U]), dtype)
    out = torch_zeros((M, H), dtype)
    dl.rnn_cell_forward(dtype, act, M, Kx, H, H, to_dev(xs[0], dtype), to_dev(h0, dtype), WU,
                        to_dev(b, dtype), out)
    sync()
    ref = oracle.rnn_forward(_spec(wl), xs, h0, W, U, b)[1]
    assert rel_l2(to_np(out), ref) <= TOL[dtype]
    assert out.device == dev


@pytest.mark.parametrize("dtype,cfg", [("f32", c) for c in (0, 1, 3, 4, 5)] +
                         [("bf16", c) for c in (0, 1, 3, 4, 10, 11, 12, 13, 14, 16, 17, 18, 19)])
def test_cell_forward_every_configuration(dtype, cfg, monkeypatch):
    """Each tile configuration forced on a two-phase product whose phases both
    end inside a k-tile and whose rows and columns are ragged (a configuration
    that cannot run a two-phase product, 14, falls back)."""
    M, Kx, H = 300, 40, 72
    wl, (xs, h0, W, U, b, _) = _case(1, Kx, H, M, dtype, "tanh", seed=5)
    monkeypatch.setenv("DLVM_GEMM_CONFIG", str(cfg))
    out = torch_zeros((M, H), dtype)
    dl.rnn_cell_forward(dtype, "tanh", M, Kx, H, H, to_dev(xs[0], dtype), to_dev(h0, dtype),
                        to_dev(np.concatenate([W, U]), dtype), to_dev(b, dtype), out)
    sync()
    ref = oracle.rnn_forward(_spec(wl), xs, h0, W, U, b)[1]
    assert rel_l2(to_np(out), ref) <= TOL[dtype]


def torch_zeros(shape, dtype):
    import torch
    return torch.zeros(shape, dtype=torch_dtype(dtype), device=device())


def sync():
    import torch
    torch.cuda.synchronize()


def _run(wl, inputs, wrt_x, wrt_h0, B=None, use_ws=True):
    """Forward and backward on the GPU; host copies of every result."""
    import torch
    xs, h0, W, U, b, dhs = inputs
    T, Kx, H = wl.steps, wl.in_width, wl.hidden
    B = h0.shape[0] if B is None else B
    dev = device()
    m = dl.Rnn(T, Kx, H, wl.act, wl.dtype, wrt_x, wrt_h0, B)
    P = m.pack_cell(W, U, b, dev, torch_dtype(wl.dtype))
    xd = to_dev(xs, wl.dtype)
    hs = torch.full((T + 1, B, H), float("nan"), dtype=torch_dtype(wl.dtype), device=dev)
    hs[0] = to_dev(h0, wl.dtype)
    ws = torch.full((m.workspace_bytes(B),), 0xFF, dtype=torch.uint8, device=dev)
    m.forward(P, xd, B, hs, ws if use_ws else None)
    dP = torch.full((m.param_count(),), float("nan"), device=dev)
    dxs = torch.full((T, B, Kx), float("nan"), device=dev) if wrt_x else None
    dh0 = torch.full((B, H), float("nan"), device=dev) if wrt_h0 else None
    m.backward(P, xd, hs, to_dev(dhs, wl.dtype), B, dP, dxs, dh0, ws)
    sync()
    dW, dU, db = m.split_cell(dP)
    return {"hs": to_np(hs), "dW": to_np(dW), "dU": to_np(dU), "db": to_np(db),
            "dxs": None if dxs is None else to_np(dxs), "dh0": None if dh0 is None else to_np(dh0),
            "dP": dP, "model": m, "P": P}


def _compare(wl, got, inputs, wrt_x, wrt_h0, tol=None):
    xs, h0, W, U, b, dhs = inputs
    tol = TOL[wl.dtype] if tol is None else tol
    spec = _spec(wl)
    hs = oracle.rnn_forward(spec, xs, h0, W, U, b)
    # the seeds as the GPU reads them (stored in the storage type)
    dq = oracle.round_to_bf16(dhs) if wl.dtype == "bf16" else dhs
    dW, dU, db, dxs, dh0 = oracle.rnn_vjp(spec, xs, h0, W, U, b, dq, wrt_x, wrt_h0)
    np.testing.assert_array_equal(got["hs"][0], hs[0])    # h0 is the caller's
    assert rel_l2(got["hs"][1:], hs[1:]) <= tol
    for name, ref in (("dW", dW), ("dU", dU), ("db", db), ("dxs", dxs), ("dh0", dh0)):
        if ref is None:
            continue
        e = rel_l2(got[name], ref)
        assert e <= tol, (name, e)


@pytest.mark.parametrize("dtype,act,T,Kx,H,B,wrt_x,wrt_h0", [
    ("f32", "tanh", 5, 40, 72, 37, True, True),
    ("f32", "sigmoid", 4, 37, 50, 19, False, False),
    ("f32", "none", 3, 64, 64, 128, True, False),
    ("bf16", "relu", 6, 64, 128, 64, True, False),
    ("bf16", "tanh", 5, 40, 72, 300, False, True),
    ("bf16", "tanh", 1, 96, 64, 33, True, True),
])
def test_rnn_forward_backward(dtype, act, T, Kx, H, B, wrt_x, wrt_h0):
    wl, inputs = _case(T, Kx, H, B, dtype, act)
    got = _run(wl, inputs, wrt_x, wrt_h0)
    _compare(wl, got, inputs, wrt_x, wrt_h0)
    # the flat gradient's padding is zero
    import torch
    m, dP = got["model"], got["dP"]
    offs, _ = m.param_layout_lds()
    used = torch.zeros(m.param_count(), dtype=torch.bool, device=dP.device)
    used[offs[0]:offs[0] + (Kx + H) * H] = True
    used[offs[1]:offs[1] + H] = True
    assert torch.count_nonzero(dP[~used]).item() == 0


def test_r1_reduced_batch():
    """The r1 network (32 steps, 1024 -> 1024, bf16 tanh) at batch 64."""
    wl = workloads.RNN_WORKLOADS["r1"]
    inputs = workloads.make_rnn_inputs(wl, batch=64)
    got = _run(wl, inputs, True, True)
    _compare(wl, got, inputs, True, True)


def test_r1_full_batch_repeated_rows_and_sgd():
    """r1 at its full batch (1024) in the launch configuration the benchmark
    times, the batch made of 64 base rows repeated 16 times in a seeded order
    (with their seeds): every row's states and input gradients are those of
    its base row, the parameter gradient is 16 times the base one."""
    import torch
    wl = workloads.RNN_WORKLOADS["r1"]
    base = 64
    xs, h0, W, U, b, dhs = workloads.make_rnn_inputs(wl, batch=base)
    idx = workloads._rng(7, 3).permutation(np.tile(np.arange(base), wl.batch // base))
    full = (xs[:, idx], h0[idx], W, U, b, dhs[:, idx])
    got = _run(wl, full, True, True)
    spec = _spec(wl)
    hs = oracle.rnn_forward(spec, xs, h0, W, U, b)
    dW, dU, db, dxs, dh0 = oracle.rnn_vjp(spec, xs, h0, W, U, b, oracle.round_to_bf16(dhs),
                                          True, True)
    tol = TOL["bf16"]
    r = wl.batch // base
    assert rel_l2(got["hs"][1:], hs[1:, idx]) <= tol
    assert rel_l2(got["dW"], r * dW) <= tol
    assert rel_l2(got["dU"], r * dU) <= tol
    assert rel_l2(got["db"], r * db) <= tol
    assert rel_l2(got["dxs"], dxs[:, idx]) <= tol
    assert rel_l2(got["dh0"], dh0[idx]) <= tol
    # the fused update of the flat buffer (float32 master, bf16 shadow)
    m, P = got["model"], got["P"]
    master = m.pack_cell(W, U, b, device(), torch.float32)
    m.sgd_step(P, master, got["dP"], wl.lr)
    sync()
    mW, mU, mb = m.split_cell(master)
    gW, gU, gb = got["dW"], got["dU"], got["db"]
    assert rel_l2(to_np(mW), oracle.sgd_f32(W, gW, wl.lr)) <= 1e-5
    assert rel_l2(to_np(mU), oracle.sgd_f32(U, gU, wl.lr)) <= 1e-5
    assert rel_l2(to_np(mb), oracle.sgd_f32(b, gb, wl.lr)) <= 1e-5
    assert torch.equal(P, master.to(torch.bfloat16))


def test_rnn_backward_is_deterministic():
    wl, inputs = _case(8, 256, 256, 512, "bf16", "tanh")
    a = _run(wl, inputs, True, True)
    b = _run(wl, inputs, True, True)
    for k in ("hs", "dW", "dU", "db", "dxs", "dh0"):
        np.testing.assert_array_equal(a[k], b[k])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("splits", [2, 4])
@pytest.mark.parametrize("H", [512, 480])
def test_split_cell_and_recurrent_products(dtype, splits, H, monkeypatch):
    """The cell products and recurrent adjoints computed in k-slices (forced),
    summed in slice order with the epilogue (bias + activation, residual +
    act') applied after the sum; the cell's slices fall on its phase boundary
    (with H = 480 the second phase ends inside a k-tile, and rows and columns
    are ragged). Two runs are bitwise equal."""
    monkeypatch.setenv("DLVM_GEMM_SPLITS", str(splits))
    wl, inputs = _case(4, 512, H, 100, dtype, "tanh", seed=21)
    m = dl.Rnn(4, 512, H, "tanh", dtype, True, True, 100)
    names = [p["name"] for p in m.plan(100)]
    assert any(n.startswith("gemm_nn") and n.endswith(f"s{splits}") for n in names)
    assert names.count("split_epilogue") >= 4
    got = _run(wl, inputs, True, True)
    _compare(wl, got, inputs, True, True)
    again = _run(wl, inputs, True, True)
    for k in ("hs", "dW", "dU", "db", "dxs", "dh0"):
        np.testing.assert_array_equal(got[k], again[k])


def test_forward_without_workspace_matches_split_forward():
    """dlvm_rnn_forward without a workspace runs every cell product unsplit; the
    states agree with the split forward to the storage precision."""
    wl = workloads.RNN_WORKLOADS["r1"]
    inputs = workloads.make_rnn_inputs(wl, batch=128)
    a = _run(wl, inputs, False, False, use_ws=True)
    b = _run(wl, inputs, False, False, use_ws=False)
    assert rel_l2(a["hs"], b["hs"]) <= 1e-2
    _compare(wl, b, inputs, False, False)


@pytest.mark.parametrize("dtype,act,T,Kx,H,B", [
    ("f32", "tanh", 3, 1, 1, 1),      # one input, one unit, one row
    ("f32", "relu", 2, 3, 5, 2),
    ("bf16", "sigmoid", 4, 2, 3, 5),
    ("bf16", "tanh", 2, 8, 8, 1),
])
def test_rnn_degenerate_sizes(dtype, act, T, Kx, H, B):
    wl, inputs = _case(T, Kx, H, B, dtype, act, seed=33)
    got = _run(wl, inputs, True, True)
    _compare(wl, got, inputs, True, True)
