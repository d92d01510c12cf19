"""GPU parity of each hot-path step on its own, through the C ABI, against the oracle.

Shapes span several tiles with ragged tails, the degenerate single-row and
ten-class cases of Fig. 3, and the workloads' own layer shapes.
"""
import numpy as np
import pytest

import oracle
import paper_1711_03016_amd as dl
from helpers import TOL, assert_close, device, quant, rel_l2, to_dev, to_np

pytestmark = pytest.mark.gpu

ACTS = ["none", "sigmoid", "tanh", "relu"]
# (M, N, K): Fig. 3 (1 x 784 -> 10), small and ragged tiles, workload layers.
FWD_SHAPES = [(1, 10, 784), (16, 32, 64), (17, 33, 65), (100, 10, 512), (256, 512, 784),
              (129, 1000, 1000), (300, 130, 1024), (1025, 96, 40), (640, 520, 264)]


def _rng(*key):
    return np.random.default_rng(list(key))


def _sync():
    import torch
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype,out_dtype", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")])
@pytest.mark.parametrize("shape", FWD_SHAPES)
def test_dense_forward(dtype, out_dtype, shape):
    import torch
    M, N, K = shape
    r = _rng(1, M, N, K)
    X = r.standard_normal((M, K)).astype(np.float32)
    W = (r.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    b = r.uniform(-0.5, 0.5, N).astype(np.float32)
    for act in ACTS:
        H = torch.empty((M, N), dtype=torch.float32 if out_dtype == "f32" else torch.bfloat16,
                        device=device())
        dl.dense_forward(dtype, out_dtype, act, M, N, K, 0.75, to_dev(X, dtype), to_dev(W, dtype),
                         to_dev(b, dtype), H)
        _sync()
        ref = oracle.dense_forward(quant(X, dtype), quant(W, dtype), quant(b, dtype), act, 0.75)
        assert_close(to_np(H), ref, TOL[dtype], act)


@pytest.mark.parametrize("dtype,out_dtype", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")])
@pytest.mark.parametrize("shape", [(1, 10, 784), (16, 10, 32), (33, 17, 70), (256, 512, 512),
                                   (300, 1000, 136), (129, 64, 1000)])
def test_dense_backward_data(dtype, out_dtype, shape):
    """dX = (dY.W^T + R) * act'(u) with act' taken from the saved output act(u)."""
    import torch
    M, N, K = shape
    r = _rng(2, M, N, K)
    u = r.standard_normal((M, K)).astype(np.float32)
    W = (r.standard_normal((K, N)) / np.sqrt(N)).astype(np.float32)
    dY = (r.standard_normal((M, N)) * 0.1).astype(np.float32)
    R = (r.standard_normal((M, K)) * 0.05).astype(np.float32)
    tdt = torch.float32 if out_dtype == "f32" else torch.bfloat16
    for act in ACTS:
        for use_r in (False, True):
            Hprev = oracle.apply_act(quant(u, "f32"), act).astype(np.float32)
            dX = torch.empty((M, K), dtype=tdt, device=device())
            Rd = to_dev(R, out_dtype) if use_r else None
            dl.dense_backward_data(dtype, out_dtype, act, M, N, K, to_dev(dY, dtype),
                                   to_dev(W, dtype), to_dev(Hprev, dtype), Rd, dX)
            _sync()
            ref = oracle.dense_vjp_input(quant(u, "f32"), quant(W, dtype), quant(dY, dtype), act)
            if use_r:
                ref = ref + (quant(R, out_dtype) if out_dtype == "bf16" else R)
            assert_close(to_np(dX), ref, TOL[dtype], (act, use_r))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 10, 784), (16, 32, 64), (16, 10, 32), (37, 129, 66),
                                   (256, 512, 784), (256, 10, 512), (4096, 10, 1024),
                                   (1000, 136, 72)])
def test_dense_backward_params(dtype, shape):
    """dW = X^T.dY (float32) and db = column sums of dY (float32)."""
    import torch
    M, N, K = shape
    r = _rng(3, M, N, K)
    X = r.standard_normal((M, K)).astype(np.float32)
    dY = (r.standard_normal((M, N)) * 0.01).astype(np.float32)
    dW = torch.empty((K, N), dtype=torch.float32, device=device())
    db = torch.empty((N,), dtype=torch.float32, device=device())
    dl.dense_backward_params(dtype, M, N, K, to_dev(X, dtype), to_dev(dY, dtype), dW, db)
    _sync()
    rdW, rdb = oracle.dense_vjp_params(quant(X, dtype), quant(dY, dtype))
    assert_close(to_np(dW), rdW, TOL[dtype] / 10, "dW", row_tol=TOL[dtype])
    assert_close(to_np(db), rdb, TOL[dtype] / 10, "db", row_tol=TOL[dtype])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("rows,classes", [(1, 10), (16, 10), (256, 10), (1000, 1000), (4097, 10),
                                          (33, 3), (70, 65), (2048, 1000)])
def test_softmax_xent(dtype, rows, classes):
    import torch
    r = _rng(4, rows, classes)
    z = (r.standard_normal((rows, classes)) * 3).astype(np.float32)
    y = r.integers(0, classes, rows).astype(np.int32)
    ws = torch.zeros(dl.softmax_xent_ws_bytes(rows), dtype=torch.uint8, device=device())
    dz = torch.empty((rows, classes), dtype=torch.float32 if dtype == "f32" else torch.bfloat16,
                     device=device())
    loss = torch.empty(1, dtype=torch.float32, device=device())
    yd = torch.from_numpy(y).to(device())
    dl.softmax_xent(dtype, rows, classes, to_dev(z), yd, 1.0 / rows, dz, loss, ws)
    _sync()
    rl, rdz = oracle.softmax_xent(z.astype(np.float64), y)
    assert abs(loss.item() - rl) <= 1e-5 * abs(rl)
    got = to_np(dz)
    assert_close(got, rdz, TOL[dtype], "dlogits")
    # labels are handled exactly: the one negative entry of each row is at its label
    neg = got < 0
    assert (neg.sum(axis=1) == 1).all()
    np.testing.assert_array_equal(np.argmax(neg, axis=1), y)
    assert torch.equal(yd.cpu(), torch.from_numpy(y))  # labels are never written


def test_softmax_xent_label_out_of_range():
    import torch
    rows, classes = 64, 10
    r = _rng(5)
    z = r.standard_normal((rows, classes)).astype(np.float32)
    y = r.integers(0, classes, rows).astype(np.int32)
    m = dl.Model((4, classes), ("none",), batch_max=rows)
    ws = torch.zeros(dl.softmax_xent_ws_bytes(rows), dtype=torch.uint8, device=device())
    dz = torch.empty((rows, classes), device=device())
    loss = torch.empty(1, device=device())
    for bad in (classes, -1):
        yb = y.copy()
        yb[7] = bad
        dl.softmax_xent("f32", rows, classes, to_dev(z), torch.from_numpy(yb).to(device()),
                        1.0 / rows, dz, loss, ws)
        assert m.check(ws) == dl.ERR_LABEL_RANGE
        assert np.isnan(loss.item())
    dl.softmax_xent("f32", rows, classes, to_dev(z), torch.from_numpy(y).to(device()),
                    1.0 / rows, dz, loss, ws)
    assert m.check(ws) == dl.OK


@pytest.mark.parametrize("rows,cols", [(5, 7), (17, 36), (64, 4096), (333, 1000)])
def test_chain8(rows, cols):
    import torch
    r = _rng(6, rows, cols)
    z = (r.standard_normal((rows, cols)) * 0.5).astype(np.float32)
    b = (r.standard_normal(cols) * 0.2).astype(np.float32)
    xs = r.standard_normal((rows, cols)).astype(np.float32)
    ws = torch.zeros(dl.chain8_ws_bytes(rows, cols), dtype=torch.uint8, device=device())
    zb = torch.empty((rows, cols), device=device())
    xb = torch.empty((rows, cols), device=device())
    loss = torch.empty(1, device=device())
    dl.chain8(rows, cols, to_dev(z), to_dev(b), to_dev(xs), zb, xb, loss, ws)
    _sync()
    rl, rdz, _, rdx, _ = oracle.chain8(z.astype(np.float64), b.astype(np.float64),
                                       xs.astype(np.float64))
    assert abs(loss.item() - rl) <= 1e-5 * rl
    assert_close(to_np(zb), rdz, TOL["f32"], "zbar")
    assert_close(to_np(xb), rdx, TOL["f32"], "xbar")


def test_chain8_full_size():
    """The chain at the stress workload's size (8192 x 4096), every element checked.

    The oracle runs on row blocks: rows are independent and the mean's seed
    1/(rows cols) only rescales each block's adjoint.
    """
    import torch
    rows, cols = 8192, 4096
    r = _rng(7)
    z = (r.standard_normal((rows, cols), dtype=np.float32) / 64).astype(np.float32)
    b = (r.standard_normal(cols) * 0.1).astype(np.float32)
    xs = (r.standard_normal((rows, cols), dtype=np.float32) / 64).astype(np.float32)
    ws = torch.zeros(dl.chain8_ws_bytes(rows, cols), dtype=torch.uint8, device=device())
    zb = torch.empty((rows, cols), device=device())
    xb = torch.empty((rows, cols), device=device())
    loss = torch.empty(1, device=device())
    dl.chain8(rows, cols, to_dev(z), to_dev(b), to_dev(xs), zb, xb, loss, ws)
    _sync()
    gz, gx = to_np(zb), to_np(xb)
    blk = 1024
    tot = 0.0
    num_z = den_z = num_x = den_x = 0.0
    for r0 in range(0, rows, blk):
        sl = slice(r0, r0 + blk)
        l, dz, _, dx, _ = oracle.chain8(z[sl].astype(np.float64), b.astype(np.float64),
                                        xs[sl].astype(np.float64))
        s = blk / rows
        tot += l * s
        dz *= s
        dx *= s
        num_z += np.sum((gz[sl] - dz) ** 2); den_z += np.sum(dz ** 2)
        num_x += np.sum((gx[sl] - dx) ** 2); den_x += np.sum(dx ** 2)
    assert abs(loss.item() - tot) <= 1e-5 * tot
    assert np.sqrt(num_z / den_z) <= TOL["f32"]
    assert np.sqrt(num_x / den_x) <= TOL["f32"]


@pytest.mark.parametrize("n", [1, 7, 4099, 1 << 20])
def test_sgd(n):
    import torch
    r = _rng(8, n)
    p = r.standard_normal(n).astype(np.float32)
    g = r.standard_normal(n).astype(np.float32)
    lr = 0.01
    pd = to_dev(p)
    dl.sgd("f32", n, pd, None, to_dev(g), lr)
    _sync()
    ref = oracle.sgd_f32(p, g, lr)
    got = pd.cpu().numpy()
    ulp = np.spacing(np.abs(ref))
    assert (np.abs(got.astype(np.float64) - ref) <= ulp).all()
    # bf16 shadow of a float32 master
    master = to_dev(p)
    shadow = torch.empty(n, dtype=torch.bfloat16, device=device())
    dl.sgd("bf16", n, shadow, master, to_dev(g), lr)
    _sync()
    rm, rs = oracle.sgd_bf16(p, g, lr)
    gm = master.cpu().numpy().astype(np.float64)
    assert (np.abs(gm - rm) <= np.spacing(np.abs(rm))).all()
    gs = to_np(shadow)
    mism = gs != rs
    # a master one ulp apart may round to the neighbouring bf16 value
    assert mism.sum() <= max(1, n // 10000)
    if mism.any():
        assert (np.abs(gs - rs)[mism] <= np.abs(rs[mism]) * 2.0 ** -7).all()


def test_host_errors_enqueue_nothing():
    import torch
    X = torch.zeros((4, 8), device=device())
    W = torch.zeros((8, 4), device=device())
    H = torch.zeros((4, 4), device=device())
    with pytest.raises(dl.DlvmError) as e:
        dl.dense_forward("f32", "bf16", "none", 4, 4, 8, 1.0, X, W, None, H)
    assert e.value.status == dl.ERR_UNSUPPORTED
    with pytest.raises(dl.DlvmError) as e:
        dl.dense_forward("f32", "f32", "none", 4, 4, 8, 1.0, X.data_ptr() + 4, W, None, H)
    assert e.value.status == dl.ERR_MISALIGNED
    with pytest.raises(dl.DlvmError) as e:
        dl.dense_forward("f32", "f32", "none", 0, 4, 8, 1.0, X, W, None, H)
    assert e.value.status == dl.ERR_INVALID_ARG
